"""CPU oracle for the Sparse DNN Challenge inference (Kepner et al., 2019) -- TEST INFRASTRUCTURE.

Only tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import this
package. The product path (``paper_1909_05631_amd``) never imports it.

The arithmetic lives in ``oracle.c`` (fp32, ascending-source fused multiply-add chains, Sec. II
batched equation and the Sec. V serial loop); this module only loads it and marshals arrays.
Every function of the oracle is pinned by the ``-m "not gpu"`` tests in ``tests/test_oracle*.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    src = os.path.join(_HERE, "oracle.c")
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                               "-o", tmp, src, "-lm", "-lpthread"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.oracle_create.argtypes = [i32, i64, ctypes.c_float, vp]
        L.oracle_create.restype = vp
        L.oracle_destroy.argtypes = [vp]
        L.oracle_destroy.restype = None
        L.oracle_layer.argtypes = [vp, vp, vp, vp, vp, i32]
        L.oracle_layer.restype = ctypes.c_int
        L.oracle_num_layers.argtypes = [vp]
        L.oracle_num_layers.restype = i64
        L.oracle_live_count.argtypes = [vp]
        L.oracle_live_count.restype = i64
        L.oracle_live_counts.argtypes = [vp, vp]
        L.oracle_live_counts.restype = None
        L.oracle_categories.argtypes = [vp, vp]
        L.oracle_categories.restype = i64
        L.oracle_rows.argtypes = [vp, vp, i64, vp]
        L.oracle_rows.restype = None
        L.oracle_margin.argtypes = [vp, vp]
        L.oracle_margin.restype = ctypes.c_double
        L.oracle_min_final_rowmax.argtypes = [vp]
        L.oracle_min_final_rowmax.restype = ctypes.c_double
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """Inference state for a batch of input rows; apply layers one at a time."""

    def __init__(self, y0: np.ndarray, ymax: float = 32.0):
        y0 = np.ascontiguousarray(y0, dtype=np.float32)
        if y0.ndim != 2:
            raise ValueError("y0 must be (rows, neurons)")
        self.m, self.n = y0.shape
        self._y0 = y0
        self._h = lib().oracle_create(self.n, self.m, ymax, _p(y0))
        if not self._h:
            raise ValueError("oracle_create rejected its arguments")

    def close(self):
        if self._h:
            lib().oracle_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def layer(self, col_ptr: np.ndarray, row_idx: np.ndarray, val: np.ndarray, bias: np.ndarray,
              threads: int = 1) -> None:
        col_ptr = np.ascontiguousarray(col_ptr, dtype=np.int64)
        row_idx = np.ascontiguousarray(row_idx, dtype=np.int32)
        val = np.ascontiguousarray(val, dtype=np.float32)
        bias = np.ascontiguousarray(bias, dtype=np.float32)
        if col_ptr.shape != (self.n + 1,) or bias.shape != (self.n,):
            raise ValueError("layer shapes do not match the network width")
        if col_ptr[-1] > row_idx.size or col_ptr[-1] > val.size:
            raise ValueError("col_ptr runs past the index/value arrays")
        rc = lib().oracle_layer(self._h, _p(col_ptr), _p(row_idx), _p(val), _p(bias), threads)
        if rc != 0:
            raise ValueError(f"oracle_layer failed ({rc})")

    @property
    def num_layers(self) -> int:
        return int(lib().oracle_num_layers(self._h))

    @property
    def live(self) -> int:
        return int(lib().oracle_live_count(self._h))

    def live_counts(self) -> np.ndarray:
        out = np.empty(self.num_layers + 1, dtype=np.int64)
        lib().oracle_live_counts(self._h, _p(out))
        return out

    def categories(self) -> np.ndarray:
        n = lib().oracle_categories(self._h, None)
        ids = np.empty(max(n, 1), dtype=np.int64)
        lib().oracle_categories(self._h, _p(ids))
        return ids[:n]

    def rows(self, ids) -> np.ndarray:
        ids = np.ascontiguousarray(ids, dtype=np.int64)
        if ids.size and (ids.min() < 0 or ids.max() >= self.m):
            raise IndexError("row id out of range")
        out = np.empty((ids.size, self.n), dtype=np.float32)
        lib().oracle_rows(self._h, _p(ids), ids.size, _p(out))
        return out

    def margin(self) -> tuple[float, np.ndarray]:
        """(min |z + b| over every layer applied so far and every entry with z != 0, the same per
        row); +inf where no such entry was seen."""
        per = np.empty(max(self.m, 1), dtype=np.float64)
        m = lib().oracle_margin(self._h, _p(per))
        return float(m), per[: self.m]

    def min_final_rowmax(self) -> float:
        """Smallest row maximum of the current Y over the rows that are categories (+inf if none)."""
        return float(lib().oracle_min_final_rowmax(self._h))


def run(y0: np.ndarray, layers, ymax: float = 32.0, threads: int = 1) -> Oracle:
    """Apply every (col_ptr, row_idx, val, bias) in `layers` in order and return the state."""
    o = Oracle(y0, ymax)
    for (cp, ri, v, b) in layers:
        o.layer(cp, ri, v, b, threads)
    return o


def run_config_layers(y0: np.ndarray, net_id: int, n_layers: int, n: int, k: int, weight: float, bias_value: float,
                      ymax: float = 32.0, threads: int = 1, chunk: int = 8, stop_when_dead: bool = True) -> Oracle:
    """Stream the seeded layers of network `net_id` through the oracle, `chunk` layers at a time.

    When every row is dead the remaining layers cannot change anything (Z = 0 stays 0), so with
    stop_when_dead the loop ends early; the live counts of the skipped layers are all zero."""
    import synth  # the input generator; holds none of the inference arithmetic

    o = Oracle(y0, ymax)
    bias = np.full(n, bias_value, dtype=np.float32)
    l = 0
    while l < n_layers:
        if stop_when_dead and o.live == 0:
            break
        nl = min(chunk, n_layers - l)
        cp, ri, v = synth.layers_csc(net_id, l, nl, n, k, weight)
        for i in range(nl):
            o.layer(cp[i], ri, v, bias, threads)
            if stop_when_dead and o.live == 0:
                break
        l += nl
    return o


def padded_live_counts(o: Oracle, n_layers: int) -> np.ndarray:
    """Live counts for all n_layers+1 boundaries, zeros after an early stop."""
    c = o.live_counts()
    out = np.zeros(n_layers + 1, dtype=np.int64)
    out[: c.size] = c
    return out
