"""Helpers for GPU parity tests: run the HIP library through its C ABI and the oracle side by side on
the same seeded inputs."""
from __future__ import annotations

import sys
import time

import numpy as np

import oracle
import synth


def log(msg: str) -> None:
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU test needs a GPU")
    return torch


class GpuNet:
    """One libsdnn network with its device buffers (torch memory) for a given input batch."""

    def __init__(self, n: int, n_layers: int, ymax: float = 32.0, equal_values: bool = False):
        from paper_1909_05631_amd import sdnn
        self.torch = torch_cuda()
        self.net = sdnn.Net(n, n_layers, ymax, equal_value_kernels=equal_values)
        self.n, self.n_layers = n, n_layers

    def load(self, l0, cp, ri, v, b):
        self.net.load_layers(l0, cp, ri, v, b)

    def load_config_layers(self, net_id, k=32, weight=1.0 / 16.0, bias_value=None, chunk=32):
        l = 0
        while l < self.n_layers:
            nl = min(chunk, self.n_layers - l)
            cp, ri, v = synth.layers_csc(net_id, l, nl, self.n, k, weight)
            self.net.load_layers(l, cp, ri, v, np.full((nl, self.n), bias_value, np.float32))
            l += nl

    def run(self, y0: np.ndarray, y0_dev=None):
        torch = self.torch
        m = y0.shape[0] if y0 is not None else y0_dev.shape[0]
        if y0_dev is None:
            y0_dev = torch.from_numpy(np.ascontiguousarray(y0, np.float32)).cuda()
        nb = self.net.workspace_bytes(m)
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
        self.net.infer(y0_dev, m, ws, nb, torch.cuda.current_stream())
        cats = self.net.categories()
        self._keep = (ws, y0_dev)
        return cats


def oracle_run(y0, layers, ymax=32.0, threads=8):
    return oracle.run(y0, layers, ymax, threads)


def assert_parity(gpu: GpuNet, o: oracle.Oracle, cats: np.ndarray, check_rows=True, rel_tol=1e-5):
    """Categories and live counts exactly; surviving rows within rel_tol (fp32 values; the canonical
    order makes them bit-identical, which is asserted too)."""
    ocats = o.categories()
    np.testing.assert_array_equal(cats, ocats)
    counts = gpu.net.live_counts()
    oc = oracle.padded_live_counts(o, gpu.n_layers)
    np.testing.assert_array_equal(counts, oc)
    if check_rows and ocats.size:
        g = gpu.net.final_rows(ocats)
        r = o.rows(ocats)
        np.testing.assert_allclose(g, r, rtol=rel_tol, atol=0)
        np.testing.assert_array_equal(g, r)
