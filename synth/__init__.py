"""Seeded synthetic workloads for the Sparse DNN Challenge (Kepner et al., 2019).

Inputs only: weight-layer patterns (CSC), bias tables and binary input images. Nothing here computes
any part of the inference; the CPU oracle and the GPU library both consume these arrays.

The configurations follow the paper's network sizes (Table 1: neurons, 32 connections per neuron,
bias per size; Table 2: layer counts) with synthetic stand-ins for the missing RadiX-Net networks
and MNIST-derived inputs (Sec. IV): random permutation-union layers and seeded stroke images.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

ROOT_SEED = 190905631
_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile libsynth.so with gcc (host code only)."""
    src = os.path.join(_HERE, "synth.c")
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                               "-o", tmp, src, "-lpthread"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        L = ctypes.CDLL(_LIB_PATH)
        u64, i32, i64 = ctypes.c_uint64, ctypes.c_int32, ctypes.c_int64
        vp = ctypes.c_void_p
        L.synth_layers_csc.argtypes = [u64, u64, i32, i32, i32, i32, ctypes.c_float, vp, vp, vp, i32]
        L.synth_layers_csc.restype = ctypes.c_int
        L.synth_layer_perms.argtypes = [u64, u64, u64, i32, i32, vp]
        L.synth_layer_perms.restype = ctypes.c_int
        L.synth_radix_layers_csc.argtypes = [u64, u64, i32, i32, i32, ctypes.c_float, vp, vp, vp, i32]
        L.synth_radix_layers_csc.restype = ctypes.c_int
        L.synth_radix_perm.argtypes = [u64, u64, u64, i32, vp]
        L.synth_radix_perm.restype = ctypes.c_int
        L.synth_inputs.argtypes = [u64, u64, i32, i32, i64, i64, ctypes.c_double, ctypes.c_double, vp, i32]
        L.synth_inputs.restype = ctypes.c_int
        L.synth_stream_value.argtypes = [u64, u64]
        L.synth_stream_value.restype = u64
        L.synth_mix64.argtypes = [u64]
        L.synth_mix64.restype = u64
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def default_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


@dataclass(frozen=True)
class Config:
    """One workload: network size, depth, input count and the Table 1 bias."""
    name: str
    net_id: int
    input_set: int
    n_rows: int
    n_neurons: int
    n_layers: int
    bias: float
    k: int = 32
    ymax: float = 32.0
    weight: float = 1.0 / 16.0
    density_mean: float = 0.19
    density_sd: float = 0.05

    @property
    def side(self) -> int:
        r = int(round(self.n_neurons ** 0.5))
        assert r * r == self.n_neurons
        return r

    @property
    def nnz_per_layer(self) -> int:
        return self.n_neurons * self.k

    @property
    def total_nnz(self) -> int:
        return self.nnz_per_layer * self.n_layers


# Table 1 biases; Table 2 depths; 60,000 inputs as in Sec. IV (2,000 for the small case).
CONFIGS = [
    Config("n1024-l120-m2000", net_id=1, input_set=1, n_rows=2000, n_neurons=1024, n_layers=120, bias=-0.30),
    Config("n1024-l120-m60000", net_id=1, input_set=1, n_rows=60000, n_neurons=1024, n_layers=120, bias=-0.30),
    Config("n4096-l480-m60000", net_id=2, input_set=2, n_rows=60000, n_neurons=4096, n_layers=480, bias=-0.35),
    Config("n16384-l1920-m60000", net_id=3, input_set=3, n_rows=60000, n_neurons=16384, n_layers=1920, bias=-0.40),
    Config("n65536-l1920-m60000", net_id=4, input_set=4, n_rows=60000, n_neurons=65536, n_layers=1920, bias=-0.45),
]


def layers_csc(net_id: int, l0: int, nl: int, n: int, k: int = 32, weight: float = 1.0 / 16.0,
               root: int = ROOT_SEED, threads: int | None = None):
    """Layers [l0, l0+nl) as one CSC chunk: col_ptr (nl, n+1) int64 with offsets continuing across
    layers, row_idx (nl*n*k,) int32 sorted ascending within each column, val (nl*n*k,) float32."""
    col_ptr = np.empty((nl, n + 1), dtype=np.int64)
    row_idx = np.empty(nl * n * k, dtype=np.int32)
    val = np.empty(nl * n * k, dtype=np.float32)
    rc = lib().synth_layers_csc(root, net_id, l0, nl, n, k, weight, _ptr(col_ptr), _ptr(row_idx), _ptr(val),
                                threads or default_threads())
    if rc != 0:
        raise RuntimeError(f"synth_layers_csc failed ({rc})")
    return col_ptr, row_idx, val


def layer_perms(net_id: int, layer: int, n: int, k: int = 32, root: int = ROOT_SEED) -> np.ndarray:
    """The k permutations (k, n) whose union is layer `layer`: W(i, perm[a, i]) != 0."""
    perm = np.empty((k, n), dtype=np.int32)
    rc = lib().synth_layer_perms(root, net_id, layer, n, k, _ptr(perm))
    if rc != 0:
        raise RuntimeError(f"synth_layer_perms failed ({rc})")
    return perm


def radix_depth(n: int) -> int:
    """D for a structured network of n = 16 * 2^D neurons (Table 1: D = 6, 8, 10, 12), else 0."""
    d = 0
    while n >= 32 and n % 16 == 0 and (1 << d) < n // 16:
        d += 1
    return d if n >= 32 and n % 16 == 0 and (1 << d) == n // 16 else 0


def radix_layers_csc(net_id: int, l0: int, nl: int, n: int, weight: float = 1.0 / 16.0, root: int = ROOT_SEED,
                     threads: int | None = None):
    """Structured (RadiX-Net style) layers [l0, l0+nl) in the layout of layers_csc with k = 32: base layer
    i of a radix-2 DNN on n / 16 nodes (node u links to u and u + 2^i), Kronecker-expanded by 16 x 16
    blocks, copy c of the D base layers relabelled by the permutation radix_perm(net_id, c, n)."""
    col_ptr = np.empty((nl, n + 1), dtype=np.int64)
    row_idx = np.empty(nl * n * 32, dtype=np.int32)
    val = np.empty(nl * n * 32, dtype=np.float32)
    rc = lib().synth_radix_layers_csc(root, net_id, l0, nl, n, weight, _ptr(col_ptr), _ptr(row_idx), _ptr(val),
                                      threads or default_threads())
    if rc != 0:
        raise RuntimeError(f"synth_radix_layers_csc failed ({rc})")
    return col_ptr, row_idx, val


def radix_perm(net_id: int, copy: int, n: int, root: int = ROOT_SEED) -> np.ndarray:
    """P_c as an array: neuron x of the base labelling is neuron perm[x] of copy `copy`."""
    perm = np.empty(n, dtype=np.int32)
    rc = lib().synth_radix_perm(root, net_id, copy, n, _ptr(perm))
    if rc != 0:
        raise RuntimeError(f"synth_radix_perm failed ({rc})")
    return perm


def inputs(set_id: int, side: int, row0: int, nrows: int, kind: str = "strokes", pa: float = 0.19,
           pb: float = 0.05, root: int = ROOT_SEED, threads: int | None = None) -> np.ndarray:
    """Binary images as dense float32 rows (nrows, side*side). kind: strokes (density mean pa, sd pb),
    bernoulli (p = pa) or mixed (density U(pa, pb) per image)."""
    kinds = {"strokes": 0, "bernoulli": 1, "mixed": 2}
    out = np.empty((nrows, side * side), dtype=np.float32)
    rc = lib().synth_inputs(root, set_id, kinds[kind], side, row0, nrows, pa, pb, _ptr(out),
                            threads or default_threads())
    if rc != 0:
        raise RuntimeError(f"synth_inputs failed ({rc})")
    return out


def bias_table(n_layers: int, n: int, value: float) -> np.ndarray:
    """Bias vectors b_l for every layer (Table 1 gives one value per network size)."""
    return np.full((n_layers, n), value, dtype=np.float32)


def config_inputs(cfg: Config, row0: int = 0, nrows: int | None = None, threads: int | None = None) -> np.ndarray:
    nrows = cfg.n_rows - row0 if nrows is None else nrows
    return inputs(cfg.input_set, cfg.side, row0, nrows, "strokes", cfg.density_mean, cfg.density_sd,
                  threads=threads)


def random_csc(rng: np.random.Generator, n: int, degrees: np.ndarray, wlo: float = -1.0, whi: float = 1.0):
    """A random single layer with the given per-column degree (sources sorted ascending), for tests.
    Values are drawn uniformly in [wlo, whi) and rounded to float32."""
    col_ptr = np.zeros(n + 1, dtype=np.int64)
    col_ptr[1:] = np.cumsum(degrees)
    rows = np.empty(int(col_ptr[-1]), dtype=np.int32)
    for j in range(n):
        d = int(degrees[j])
        rows[col_ptr[j]:col_ptr[j + 1]] = np.sort(rng.choice(n, size=d, replace=False))
    vals = rng.uniform(wlo, whi, size=rows.size).astype(np.float32)
    return col_ptr, rows, vals
