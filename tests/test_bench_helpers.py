"""Host-side pieces of bench.py: the algorithmic byte count of a layer (dense fp32 live rows, weights
once, bias) and the lookup of committed rocprofv3 records, which must ignore records taken with
another kernel source."""
import json

import numpy as np

import bench


def test_algorithmic_layer_bytes_counts_rows_weights_and_bias():
    # 4 neurons, 8 weights, 2 rows in, 1 row out: 4*4*(2+1) + 8*8 + 4*4
    assert bench.algorithmic_layer_bytes(4, 8, 2, 1) == 48 + 64 + 16
    # nothing enters: nothing moves
    assert bench.algorithmic_layer_bytes(4, 8, 0, 0) == 0
    # the n65536 network's layer 1 on the stroke inputs: 60,000 rows in, 8,103 out
    n, nnz = 65536, 32 * 65536
    assert bench.algorithmic_layer_bytes(n, nnz, 60000, 8103) == 4 * n * 68103 + 8 * nnz + 4 * n


def test_committed_records_follow_the_kernel_source(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_sha", lambda: "abc")
    rec = {"kernel": "k_layer_gfm_u8", "kernel_source_sha256": "abc", "bytes_per_launch": 123,
           "lds": {"command": "", "kernels": {"k_layer_gfm_u8<32, true, 64>": {"conflict_cycle_frac": 0.012},
                                              "k_layer_count<16, false>": {"conflict_cycle_frac": 0.48},
                                              "k_layer_gfm<32, 32, true>": {"conflict_cycle_frac": 0.03}}}}
    (tmp_path / "profiles" / "traffic_w.json").write_text(json.dumps(rec))
    assert bench.committed_traffic("w", "k_layer_gfm_u8") == 123
    assert bench.committed_traffic("w", "k_layer_gfm") is None  # another kernel's record
    assert bench.committed_lds("w", "k_layer_gfm_u8") == {"k_layer_gfm_u8<32, true, 64>": 0.012}
    assert bench.committed_lds("w", "k_pack_bits+k_layer_count") == {"k_layer_count<16, false>": 0.48}
    assert bench.committed_traffic("x", "k_layer_gfm_u8") is None  # no record
    monkeypatch.setattr(bench, "kernel_source_sha", lambda: "def")  # source changed since
    assert bench.committed_traffic("w", "k_layer_gfm_u8") is None
    assert bench.committed_lds("w", "k_layer_gfm_u8") is None


def test_more_than_one_gpu_is_refused():
    """The benchmark measures one GPU's share; asking for more exits with a message, touching no GPU."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU only" in r.stderr and r.stdout == ""


def test_workload_names():
    import synth
    c4 = synth.CONFIGS[4]
    assert bench.workload(c4, "strokes", 0) is c4
    assert bench.workload(c4, "alllive", 16).name == "alllive-n65536-l16-m60000"
    assert bench.workload(c4, "alllive", 16).total_nnz == 16 * c4.nnz_per_layer
    assert bench.workload_name(bench.workload(synth.CONFIGS[2], "strokes", 40), "radix") == "radix-n4096-l40-m60000"


def test_source_code_sha_ignores_comments_only():
    """The counter records stay valid across comment edits of the kernel source, not across code
    edits."""
    a = "int f(int x) { return x + 1; }  // one\n/* block */\n"
    b = "// header\nint f(int x) {\n  return x + 1;  /* two */\n}\n"
    c = "int f(int x) { return x + 2; }\n"
    assert bench.source_code_sha(a) == bench.source_code_sha(b)
    assert bench.source_code_sha(a) != bench.source_code_sha(c)
