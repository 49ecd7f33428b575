"""GPU parity at the full sizes of the five workloads (Table 1 widths and biases, Table 2 depths,
60,000 inputs as in Sec. IV; 2,000 for the small case), in the launch configuration the benchmark
times: every row against the oracle, with exact live counts, categories and surviving rows. The
all-live set is checked on a seeded sample of rows (its live counts are all M, checked exactly)."""
import os

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import GpuNet, assert_parity, log

pytestmark = pytest.mark.gpu

THREADS = max(1, min(16, os.cpu_count() or 1))


def gpu_config_run(cfg, equal_values=False):
    log(f"{cfg.name}: generating inputs")
    y0 = synth.config_inputs(cfg)
    gpu = GpuNet(cfg.n_neurons, cfg.n_layers, cfg.ymax, equal_values)
    log(f"{cfg.name}: loading {cfg.n_layers} layers")
    gpu.load_config_layers(cfg.net_id, cfg.k, cfg.weight, cfg.bias)
    log(f"{cfg.name}: running the GPU")
    cats = gpu.run(y0)
    log(f"{cfg.name}: {cats.size} categories; live counts {gpu.net.live_counts()[:8].tolist()}")
    return y0, gpu, cats


@pytest.mark.parametrize("ci", [0, 1, 2, 3, 4])
def test_full_config_every_row(ci):
    """Every row of the workload against the oracle (Sec. V: compare the computed categories): the
    categories, every per-layer live count and every surviving row bit for bit."""
    cfg = synth.CONFIGS[ci]
    y0, gpu, cats = gpu_config_run(cfg)
    log(f"{cfg.name}: oracle on all {cfg.n_rows} rows")
    o = oracle.run_config_layers(y0, cfg.net_id, cfg.n_layers, cfg.n_neurons, cfg.k, cfg.weight, cfg.bias,
                                 cfg.ymax, threads=THREADS)
    log(f"{cfg.name}: oracle live counts {o.live_counts()[:8].tolist()}, {o.categories().size} categories")
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("ci", [2, 4])
def test_full_config_every_row_equal_value_kernels(ci):
    """The same with the opt-in kernels that exploit the configs' equal weights and biases (layer 0
    by counts, one weight per layer): the supplementary measurement's path, on every row."""
    cfg = synth.CONFIGS[ci]
    y0, gpu, cats = gpu_config_run(cfg, equal_values=True)
    o = oracle.run_config_layers(y0, cfg.net_id, cfg.n_layers, cfg.n_neurons, cfg.k, cfg.weight, cfg.bias,
                                 cfg.ymax, threads=THREADS)
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("ci,equal_values", [(2, False), (2, True), (3, False), (3, True), (4, False)])
def test_structured_full_config_every_row(ci, equal_values):
    """The second workload: structured (RadiX-Net style) layers of the config's width and depth on the
    config's inputs, full size on the GPU, every row against the oracle. At 16384 and 65536 neurons
    the repacks after layers 1-3 write the next layer's inputs as one- or two-byte codes."""
    cfg = synth.CONFIGS[ci]
    n, L = cfg.n_neurons, cfg.n_layers
    y0 = synth.config_inputs(cfg)
    gpu = GpuNet(n, L, cfg.ymax, equal_values)
    log(f"radix-{cfg.name}: loading {L} structured layers (equal_values={equal_values})")
    for l0 in range(0, L, 64):
        nl = min(64, L - l0)
        cp, ri, v = synth.radix_layers_csc(cfg.net_id, l0, nl, n, cfg.weight)
        gpu.load(l0, cp, ri, v, np.full((nl, n), cfg.bias, np.float32))
    cats = gpu.run(y0)
    log(f"radix-{cfg.name}: {cats.size} categories; live counts {gpu.net.live_counts()[:8].tolist()}")
    o = oracle.Oracle(y0, cfg.ymax)
    bias = np.full(n, cfg.bias, np.float32)
    l = 0
    while l < L and o.live > 0:
        nl = min(64, L - l)
        cp, ri, v = synth.radix_layers_csc(cfg.net_id, l, nl, n, cfg.weight)
        for i in range(nl):
            o.layer(cp[i], ri, v, bias, THREADS)
        l += nl
    assert_parity(gpu, o, cats)
    o.close()


@pytest.mark.parametrize("ci,nl,rows", [(2, 12, 4096), (4, 6, 512)])
def test_all_live_sampled_rows(ci, nl, rows):
    """The supplementary all-live set: Bernoulli(0.6) rows on the config's network, which keep every
    row live at every layer, so each layer runs at its full shape (60,000 rows); the first nl layers.
    A seeded sample of `rows` rows is recomputed by the oracle."""
    import bench
    cfg = bench.workload(synth.CONFIGS[ci], "alllive", nl)
    n, m = cfg.n_neurons, cfg.n_rows
    y0 = bench.input_rows(cfg, "alllive", 0, m)
    gpu = GpuNet(n, nl, cfg.ymax)
    log(f"{cfg.name}: loading {nl} layers")
    gpu.load_config_layers(cfg.net_id, cfg.k, cfg.weight, cfg.bias)
    cats = gpu.run(y0)
    counts = gpu.net.live_counts()
    log(f"{cfg.name}: {cats.size} categories; live counts {counts.tolist()}")
    assert (counts == m).all() and cats.size == m
    rng = np.random.default_rng(200 + ci)
    sample = np.sort(rng.choice(m, size=rows, replace=False))
    o = oracle.run_config_layers(y0[sample], cfg.net_id, nl, n, cfg.k, cfg.weight, cfg.bias, cfg.ymax,
                                 threads=THREADS)
    assert o.categories().size == sample.size
    np.testing.assert_array_equal(gpu.net.final_rows(sample), o.rows(o.categories()))


@pytest.mark.parametrize("ci,nl,rows", [(3, 11, 512), (4, 11, 256)])
def test_encoded_layer_inputs(ci, nl, rows):
    """All-live rows on the two widest networks (60,000 rows, 32-row fp32 tiles, code tiles of 128
    and 64 rows): the inputs of layers 2-7 take more than 256 distinct values, so their encoding
    into one-byte codes overflows the dictionary and stops, and those layers gather two-byte codes
    (up to 4096 values) or fp32; from layer 8 on every entry is 32 (saturated), the one-byte
    encoding succeeds and the layers gather one-byte codes. A seeded sample of rows is recomputed by
    the oracle; every count must be the row count."""
    import bench
    from paper_1909_05631_amd import sdnn
    cfg = bench.workload(synth.CONFIGS[ci], "alllive", nl)
    n, m = cfg.n_neurons, cfg.n_rows
    y0 = bench.input_rows(cfg, "alllive", 0, m)
    gpu = GpuNet(n, nl, cfg.ymax)
    log(f"{cfg.name}: loading {nl} layers")
    gpu.load_config_layers(cfg.net_id, cfg.k, cfg.weight, cfg.bias)
    cats = gpu.run(y0)
    counts = gpu.net.live_counts()
    kinds, launches = gpu.net.layer_info()
    names = [sdnn.KERNEL_KINDS.get(int(k)) for k in kinds]
    log(f"{cfg.name}: live counts {counts.tolist()}; kernels {names}")
    assert (counts == m).all() and cats.size == m
    assert names[0] == "k_pack_bits+k_layer_bits(codes)" and names[1] == "k_layer_gfm_u8"
    assert all(k in ("k_layer_gfm", "k_layer_gfm_u16") for k in names[2:8])  # one-byte encodings overflowed
    assert "k_layer_gfm" in names[2:8]                                       # and two-byte ones too
    assert all(k == "k_layer_gfm_u8" for k in names[8:nl])                   # encoded inputs
    rng = np.random.default_rng(300 + ci)
    sample = np.sort(rng.choice(m, size=rows, replace=False))
    o = oracle.run_config_layers(y0[sample], cfg.net_id, nl, n, cfg.k, cfg.weight, cfg.bias, cfg.ymax,
                                 threads=THREADS)
    assert o.categories().size == sample.size
    np.testing.assert_array_equal(gpu.net.final_rows(sample), o.rows(o.categories()))


def test_many_rows_every_row():
    """Five times the configs' row count (300,000 inputs of the 1024-neuron, 120-layer network):
    live lists longer than one compaction pass covers; every row against the oracle."""
    cfg = synth.CONFIGS[1]
    m = 300_000
    y0 = synth.config_inputs(cfg, 0, m)
    gpu = GpuNet(cfg.n_neurons, cfg.n_layers, cfg.ymax)
    gpu.load_config_layers(cfg.net_id, cfg.k, cfg.weight, cfg.bias)
    log(f"{m} rows of {cfg.name}: running the GPU")
    cats = gpu.run(y0)
    log(f"{cats.size} categories; live counts {gpu.net.live_counts()[:8].tolist()}")
    o = oracle.run_config_layers(y0, cfg.net_id, cfg.n_layers, cfg.n_neurons, cfg.k, cfg.weight, cfg.bias,
                                 cfg.ymax, threads=THREADS)
    assert_parity(gpu, o, cats)
