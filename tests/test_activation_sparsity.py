"""How sparse the activations entering each layer are on the seeded workloads (CPU, oracle).

The layer kernels gather feature-major segments: one 128-byte load carries 32 live rows of one
source. A path that skips zero activations can only skip a load whose 32 rows are all zero; a
row-wise path (one row's nonzero inputs scattered or tested per edge) needs lanes that each walk a
different number of terms. These tests measure, on 2048 inputs of the two widest networks, the
nonzero fraction of the live rows entering layers 0-2 and the fraction of (source, 32-row tile)
segments that are zero in every row, and pin the facts the design relies on: after layer 0 the
inputs are 9-55% nonzero, and at most about 6% of the segments could be skipped."""
import numpy as np
import pytest

import oracle
import synth


def layer_inputs(ci: int, rows: int, layers: int):
    """(live rows, nonzero fraction, all-zero 32-row segment fraction) of the input of layers
    0 .. layers - 1, live rows in ascending id order as the kernels list them."""
    cfg = synth.CONFIGS[ci]
    n = cfg.n_neurons
    y0 = synth.config_inputs(cfg, 0, rows)
    o = oracle.Oracle(y0, 32.0)
    bias = np.full(n, cfg.bias, dtype=np.float32)
    cp, ri, v = synth.layers_csc(cfg.net_id, 0, layers, n)
    out = []
    for l in range(layers):
        ids = np.arange(rows) if l == 0 else o.categories()
        y = y0[ids] if l == 0 else o.rows(ids)
        y = y[np.abs(y).sum(1) > 0]
        full = y.shape[0] // 32 * 32
        seg = (y[:full].reshape(-1, 32, n) == 0).all(1).mean() if full else float("nan")
        out.append((y.shape[0], float((y != 0).mean()), float(seg)))
        o.layer(cp[l], ri, v, bias, threads=8)
    return out


@pytest.mark.parametrize("ci", [3, 4])
def test_few_all_zero_segments_after_layer0(ci):
    stats = layer_inputs(ci, 2048, 3)
    print(synth.CONFIGS[ci].name, [(r, round(d, 3), round(s, 3)) for r, d, s in stats])
    # layer 0 reads the binary images: about a fifth of the pixels are set (the stroke generator's
    # target), and hardly a segment is empty
    assert 0.17 < stats[0][1] < 0.26 and stats[0][2] < 0.02
    for rows, dens, seg in stats[1:]:
        if rows < 64:
            continue
        # later layers: live rows 9-55% nonzero; a zero-skipping gather could drop at most ~6% of
        # its segment loads (independent 32-row segments at density d are all zero with
        # probability (1 - d)^32, 4% at d = 0.093)
        assert 0.05 < dens < 0.7
        assert seg < 0.10
