"""GPU parity: the HIP library (through its C ABI) against the CPU oracle on the same seeded inputs.

Bar: categories and per-layer live counts bit-exact; surviving final activations within 1e-5
relative (fp32), and in fact bit-identical because both sides sum in the same canonical order.

Tests run the library's default kernels, which read every edge's weight and every neuron's bias
from memory; tests parametrized with `equal_values` also run the opt-in kernels that exploit layers
whose weights and biases are all equal (sdnn_enable_equal_value_kernels)."""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import GpuNet, assert_parity, log


def sdnn_kind(k):
    from paper_1909_05631_amd import sdnn
    return sdnn.KERNEL_KINDS.get(int(k))

pytestmark = pytest.mark.gpu


def random_layers(rng, n, nl, max_deg, signed=True):
    layers = []
    for _ in range(nl):
        deg = rng.integers(0, max_deg + 1, size=n)
        cp, ri, v = synth.random_csc(rng, n, deg, -1.0 if signed else 0.0, 1.0)
        v = (v * rng.choice([0.25, 1.0, 3.0])).astype(np.float32)
        b = rng.uniform(-0.6, 0.4, size=n).astype(np.float32)
        layers.append((cp, ri, v, b))
    return layers


def run_both(n, layers, y0, ymax=32.0, equal_values=False):
    gpu = GpuNet(n, len(layers), ymax, equal_values)
    for l, (cp, ri, v, b) in enumerate(layers):
        gpu.load(l, cp, ri, v, b)
    cats = gpu.run(y0)
    o = oracle.run(y0, layers, ymax, threads=4)
    return gpu, o, cats


@pytest.mark.parametrize("seed", range(24))
def test_tiny_random_networks(seed):
    """Random widths (including widths that are not multiples of 4), ragged row counts, random column
    degrees up to the width, signed weights, biases of both signs and several YMAX values."""
    rng = np.random.default_rng(seed)
    n = int(rng.choice([1, 2, 3, 5, 8, 13, 31, 32, 33, 64, 100, 257]))
    m = int(rng.integers(1, 80))
    nl = int(rng.integers(1, 7))
    ymax = float(rng.choice([1.5, 4.0, 32.0]))
    layers = random_layers(rng, n, nl, max_deg=min(n, 40))
    y0 = (rng.random((m, n)) < rng.uniform(0.2, 0.9)).astype(np.float32) * rng.uniform(0, 2, (m, n)).astype(np.float32)
    if seed % 4 == 0:
        y0[rng.random(m) < 0.3] = 0  # all-zero input rows
    if seed % 5 == 0:
        y0 -= np.float32(0.5) * (rng.random((m, n)) < 0.1)  # negative inputs
    log(f"tiny seed={seed} n={n} m={m} layers={nl}")
    gpu, o, cats = run_both(n, layers, y0, ymax)
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("equal_values", [False, True])
@pytest.mark.parametrize("n", [1024, 2048, 4096, 16384, 65536])
def test_config_networks_mixed_inputs(n, equal_values):
    """The configs' permutation-union networks (32 weights of 1/16 per column) with inputs whose
    densities straddle the survival threshold, so categories are neither empty nor full; covers both
    kernel paths and the tile sizes of every width."""
    bias = {1024: -0.30, 2048: -0.30, 4096: -0.35, 16384: -0.40, 65536: -0.45}[n]
    side = int(round(n ** 0.5)) if int(round(n ** 0.5)) ** 2 == n else None
    m = {1024: 300, 2048: 200, 4096: 150, 16384: 70, 65536: 40}[n]
    nl = {1024: 24, 2048: 16, 4096: 16, 16384: 8, 65536: 6}[n]
    if side:
        y0 = synth.inputs(20 + n % 7, side, 0, m, "mixed", 0.2, 0.7)
    else:
        y0 = (np.random.default_rng(4).random((m, n)) < np.random.default_rng(5).uniform(0.2, 0.7, (m, 1))).astype(np.float32)
    cp, ri, v = synth.layers_csc(9, 0, nl, n)
    layers = [(cp[l], ri, v, np.full(n, bias, np.float32)) for l in range(nl)]
    log(f"config-net n={n} m={m} layers={nl} equal_values={equal_values}")
    gpu, o, cats = run_both(n, layers, y0, equal_values=equal_values)
    assert 0 < cats.size < m
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("bias", [-0.30, -0.45])
def test_closed_form_and_tie_rows(bias):
    """All-ones rows follow y_{l+1} = min(32, 2 y_l + b) to exactly 32; constant rows c = -b/2 sit on
    the survival threshold, where only the ascending-order fp32 sum decides the outcome."""
    n, nl = 1024, 10
    c = np.float32(-np.float32(bias)) / np.float32(2.0)
    y0 = np.stack([np.ones(n, np.float32), np.full(n, c, np.float32), np.zeros(n, np.float32)])
    cp, ri, v = synth.layers_csc(1, 0, nl, n)
    layers = [(cp[l], ri, v, np.full(n, bias, np.float32)) for l in range(nl)]
    gpu, o, cats = run_both(n, layers, y0)
    assert_parity(gpu, o, cats)
    assert 0 in cats
    np.testing.assert_array_equal(gpu.net.final_rows([0]), np.full((1, n), 32.0, np.float32))


def test_edge_cases():
    """Empty batch, one row, one neuron, empty columns, a single layer, values clamped at YMAX."""
    rng = np.random.default_rng(11)
    # empty batch
    cp, ri, v = synth.layers_csc(1, 0, 2, 1024)
    layers = [(cp[l], ri, v, np.full(1024, -0.3, np.float32)) for l in range(2)]
    gpu, o, cats = run_both(1024, layers, np.zeros((0, 1024), np.float32))
    assert cats.size == 0 and list(gpu.net.live_counts()) == [0, 0, 0]
    # one neuron, self loop, clamp
    lay = [(np.array([0, 1], np.int64), np.array([0], np.int32), np.array([3.0], np.float32), np.array([0.5], np.float32))] * 3
    gpu, o, cats = run_both(1, lay, np.array([[1.0], [0.0], [2.0]], np.float32), ymax=10.0)
    assert_parity(gpu, o, cats)
    np.testing.assert_array_equal(gpu.net.final_rows([0, 1, 2])[:, 0], [10.0, 0.0, 10.0])
    # empty columns everywhere but one
    n = 40
    cp = np.zeros(n + 1, np.int64); cp[8:] = 3
    lay = [(cp, np.array([1, 5, 9], np.int32), np.array([1, 1, 1], np.float32), np.zeros(n, np.float32))]
    y0 = rng.random((37, n)).astype(np.float32)
    gpu, o, cats = run_both(n, lay, y0)
    assert_parity(gpu, o, cats)


def test_rerun_is_deterministic_and_batches_independent():
    """Two runs give identical results; a run on a prefix of the rows gives that prefix's results."""
    n, nl, m = 4096, 12, 130
    y0 = synth.inputs(31, 64, 0, m, "mixed", 0.3, 0.6)
    cp, ri, v = synth.layers_csc(2, 0, nl, n)
    gpu = GpuNet(n, nl)
    gpu.load(0, cp, ri, v, np.full((nl, n), -0.35, np.float32))
    a = gpu.run(y0)
    ra = gpu.net.final_rows(a)
    b = gpu.run(y0)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(ra, gpu.net.final_rows(b))
    p = gpu.run(y0[:61])
    np.testing.assert_array_equal(p, a[a < 61])


@pytest.mark.parametrize("n,seed", [(5001, 1), (12001, 2), (8192, 3)])
def test_global_tile_path_random_networks(n, seed):
    """Widths past the LDS budget use feature-major tiles in global memory (32 or 16 rows per tile);
    random degrees (including empty columns), signed weights, widths that are not multiples of 4."""
    rng = np.random.default_rng(100 + seed)
    m, nl = int(rng.integers(20, 70)), 3
    layers = random_layers(rng, n, nl, max_deg=40)
    y0 = (rng.random((m, n)) < 0.5).astype(np.float32) * rng.uniform(0, 2, (m, n)).astype(np.float32)
    log(f"global-tile n={n} m={m} layers={nl}")
    gpu, o, cats = run_both(n, layers, y0)
    assert gpu.net.kernel_path == 1
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("n,kind", [(5001, "binary"), (12001, "binary"), (40000, "binary"), (16384, "signed-zero"),
                                    (12001, "not-binary")])
def test_layer0_bit_route(n, kind):
    """Wide layers take layer 0 from bit-packed inputs when every input is 0 or 1 (32-row bit tiles up
    to 16384 neurons, 16-row tiles beyond); -0.0 counts as 0; a single other value sends layer 0 back
    to the fp32 route. Either way the result must equal the oracle's."""
    rng = np.random.default_rng(n)
    m, nl = 75, 3
    cp, ri, v = synth.layers_csc(11, 0, nl, n) if n in (16384,) else (None, None, None)
    if cp is not None:
        layers = [(cp[l], ri, v, np.full(n, -0.40, np.float32)) for l in range(nl)]
    else:
        layers = random_layers(rng, n, nl, max_deg=32, signed=False)
        layers = [(a, b_, w * np.float32(0.5), np.full(n, -0.3, np.float32)) for (a, b_, w, _) in layers]
    dens = rng.uniform(0.2, 0.8, size=(m, 1))
    y0 = (rng.random((m, n)) < dens).astype(np.float32)
    y0[5] = 0.0
    if kind == "signed-zero":
        y0[y0 == 0] = -0.0
    if kind == "not-binary":
        y0[3, 7] = 0.5
    log(f"bit route n={n} kind={kind}")
    gpu, o, cats = run_both(n, layers, y0)
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("n,m,maxdeg", [(6000, 300, 20), (6000, 60, 20), (20000, 300, 12), (6000, 100, 0)])
def test_layer0_bit_route_short_columns(n, m, maxdeg):
    """Layer 0 on the bit route when its columns hold fewer than 32 sources (the kernel's runtime
    slot loop over a narrower ELL, read as word offsets), with more than 256 rows (one-byte codes out)
    and fewer (fp32 out), at both bit-tile heights; maxdeg 0 is a layer without edges, whose outputs
    are all zero, so every row dies at once."""
    rng = np.random.default_rng(n + m + maxdeg)
    nl = 4
    layers = []
    for l in range(nl):
        hi = maxdeg if l == 0 else 32
        deg = rng.integers(0, hi + 1, size=n) if hi > 0 else np.zeros(n, dtype=np.int64)
        cp, ri, v = synth.random_csc(rng, n, deg, -0.05, 0.3)
        layers.append((cp, ri, v, rng.uniform(-0.3, -0.1, size=n).astype(np.float32)))
    y0 = (rng.random((m, n)) < rng.uniform(0.3, 0.7, size=(m, 1))).astype(np.float32)
    log(f"bit route, short columns n={n} m={m} maxdeg={maxdeg}")
    gpu, o, cats = run_both(n, layers, y0)
    kinds, _ = gpu.net.layer_info()
    assert sdnn_kind(kinds[0]).startswith("k_pack_bits+k_layer_bits")
    if maxdeg == 0:
        assert cats.size == 0 and gpu.net.live_counts()[1] == 0
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("n,m,bias,lo,hi,kind", [
    (6000, 1100, -0.40, 0.10, 0.40, "binary"),     # 1100 -> 561 -> 213 -> ... -> 7: large, then small layers
    (6000, 1100, -0.35, 0.10, 0.30, "binary"),     # every row dies by layer 4
    (6000, 1100, -0.40, 0.10, 0.40, "scaled"),     # non-binary inputs: fp32 layer 0 over 35 tiles (5 rounds)
    (9000, 900, -0.45, 0.10, 0.40, "binary"),
])
def test_global_tile_large_lists(n, m, bias, lo, hi, kind):
    """Hundreds of live rows on the global-tile path: layers of several rounds of 8 tiles, compaction
    with exact read-back, repacking of the tiles when rows die, the switch to single-round layers that
    count their own live rows, and an early exit once no row is left."""
    nl = 12
    rng = np.random.default_rng(7)
    dens = rng.uniform(lo, hi, size=(m, 1))
    y0 = (rng.random((m, n)) < dens).astype(np.float32)
    if kind == "scaled":
        y0 *= np.float32(1.25)
    cp, ri, v = synth.layers_csc(12, 0, nl, n)
    layers = [(cp[l], ri, v, np.full(n, bias, np.float32)) for l in range(nl)]
    log(f"large lists n={n} m={m} bias={bias} kind={kind}")
    gpu, o, cats = run_both(n, layers, y0)
    assert gpu.net.kernel_path == 1
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("equal_values", [False, True])
@pytest.mark.parametrize("case", ["last", "fill", "adopt-odd"])
def test_code_layer_outputs(case, equal_values):
    """The layer after a large binary layer 0 (written as dictionary codes, or by counts with
    equal_values) gathers one-byte codes and skips storing 32-row output segments
    that are zero in every row. Its tiles are then either repacked (reading only the stored segments)
    or, when the next layer or the final read-out takes them as they are, completed with zeros.
    "last": it is the last layer; "fill": it keeps nearly every row, so no repack follows; "adopt-odd":
    layer 0 leaves 1044 live rows (16 code tiles and a half, 33 fp32 tiles), so the upper half of the
    last code tile has no fp32 tile to write."""
    n, m = 6000, 1100
    nl = {"last": 2, "fill": 4, "adopt-odd": 6}[case]
    rng = np.random.default_rng(31)
    y0 = (rng.random((m, n)) < rng.uniform(0.15, 0.40, size=(m, 1))).astype(np.float32)
    if case == "adopt-odd":
        y0[rng.choice(m, 56, replace=False)] = 0.0
    cp, ri, v = synth.layers_csc(13, 0, nl, n)
    bias = [np.full(n, -0.40, np.float32) for _ in range(nl)]
    if case == "fill":
        bias[1][:] = 0.10
    layers = [(cp[l], ri, v, bias[l]) for l in range(nl)]
    log(f"code layer outputs case={case} equal_values={equal_values}")
    gpu, o, cats = run_both(n, layers, y0, equal_values=equal_values)
    kind, _ = gpu.net.layer_info()
    assert gpu.net.kernel_path == 1 and sdnn_kind(kind[1]) == "k_layer_gfm_u8"
    counts = oracle.padded_live_counts(o, nl)
    if case == "adopt-odd":
        assert counts[1] == 1044
    if case == "fill":
        assert counts[2] * 20 > counts[1] * 19
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("equal_values", [False, True])
@pytest.mark.parametrize("n,m,kind", [(1024, 3000, "uniform"), (2048, 1500, "uniform"), (4096, 700, "uniform"),
                                      (1500, 900, "random"), (1024, 600, "dying")])
def test_fused_layers(n, m, kind, equal_values):
    """Widths up to 4096: once few enough rows are live, one launch runs every remaining layer with each
    workgroup's rows kept in LDS (16, 8 or 4 rows per workgroup by width and count). "uniform": layers
    of one weight (read through 16-bit source lists with equal_values); "random": signed weights of
    random degree; "dying": every row dies inside the fused launch."""
    nl = 10
    rng = np.random.default_rng(n + m)
    if kind == "random":
        layers = random_layers(rng, n, nl, max_deg=24)
        y0 = rng.random((m, n)).astype(np.float32) * (rng.random((m, n)) < 0.3)
    else:
        cp, ri, v = synth.layers_csc(14, 0, nl, n)
        bias = -0.30 if kind != "dying" else -0.45
        layers = [(cp[l], ri, v, np.full(n, bias, np.float32)) for l in range(nl)]
        lo, hi = (0.45, 0.7) if kind != "dying" else (0.25, 0.35)
        y0 = (rng.random((m, n)) < rng.uniform(lo, hi, size=(m, 1))).astype(np.float32)
    log(f"fused layers n={n} m={m} kind={kind} equal_values={equal_values}")
    gpu, o, cats = run_both(n, layers, y0, equal_values=equal_values)
    kinds, launches = gpu.net.layer_info()
    assert gpu.net.kernel_path == 0
    fused = [l for l in range(nl) if sdnn_kind(kinds[l]) == "k_layers_lds"]
    assert fused and launches[fused[0]] == 1 and all(launches[l] == 0 for l in fused[1:])
    assert fused == list(range(fused[0], nl))
    if kind == "dying":
        assert oracle.padded_live_counts(o, nl)[-1] == 0
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("equal_values", [False, True])
@pytest.mark.parametrize("n,kind", [(6000, "binary"), (5003, "binary"), (6000, "one-value")])
def test_counting_layer0(n, kind, equal_values):
    """Layer 0 of a uniform network on more than 256 binary rows: with equal_values by counts of the
    bit-packed inputs, by default from the bit tiles with each edge's weight, written as dictionary
    codes; at widths that are and are not multiples of 4. "one-value": a single input of 0.5 rules
    the bit route out, and layer 0 runs on fp32 tiles."""
    m, nl = 700, 4
    rng = np.random.default_rng(n)
    y0 = (rng.random((m, n)) < rng.uniform(0.2, 0.6, size=(m, 1))).astype(np.float32)
    y0[11] = 0.0
    if kind == "one-value":
        y0[300, 17] = 0.5
    cp, ri, v = synth.layers_csc(15, 0, nl, n)
    layers = [(cp[l], ri, v, np.full(n, -0.35, np.float32)) for l in range(nl)]
    log(f"counting layer 0 n={n} kind={kind} equal_values={equal_values}")
    gpu, o, cats = run_both(n, layers, y0, equal_values=equal_values)
    kinds, _ = gpu.net.layer_info()
    bits = "k_pack_bits+k_layer_count" if equal_values else "k_pack_bits+k_layer_bits(codes)"
    expect = bits if kind == "binary" else "k_layer_gfm"
    assert sdnn_kind(kinds[0]) == expect
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("kind", ["binary", "one-value"])
def test_counting_layer0_lds_widths(kind):
    # the counting route exists only with the equal-value kernels
    """Widths staged in LDS, from 2^24 inputs: layer 0 of a uniform network goes by counts of the
    bit-packed rows and is written back as fp32 rows (one mask bit per list position), then the
    row tiles take over. "one-value": an input of 0.5 keeps layer 0 on the fp32 kernel."""
    n, m, nl = 1024, 16384, 4
    rng = np.random.default_rng(77)
    y0 = (rng.random((m, n)) < rng.uniform(0.15, 0.6, size=(m, 1))).astype(np.float32)
    y0[5] = 0.0
    if kind == "one-value":
        y0[9000, 3] = 0.5
    cp, ri, v = synth.layers_csc(16, 0, nl, n)
    layers = [(cp[l], ri, v, np.full(n, -0.30, np.float32)) for l in range(nl)]
    log(f"counting layer 0 on LDS widths kind={kind}")
    gpu, o, cats = run_both(n, layers, y0, equal_values=True)
    kinds, _ = gpu.net.layer_info()
    assert gpu.net.kernel_path == 0
    assert sdnn_kind(kinds[0]) == ("k_pack_bits+k_layer_count" if kind == "binary" else "k_layer_lds")
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("m", [40, 200])
def test_few_tile_tail_dies(m):
    """Widths gathered from global tiles with few rows (at most 8 tiles per layer): every row stays
    live up to layer 20, whose bias kills them all. The few-tile launches report liveness through
    per-workgroup partial words and the host follows them through the progress word, so it must stop
    enqueuing within a few layers of the last live one; layers enqueued after it must store nothing
    and report no row (their inputs are zero)."""
    n, nl, die = 6000, 200, 20
    rng = np.random.default_rng(m)
    y0 = (rng.random((m, n)) < 0.5).astype(np.float32)
    cp, ri, v = synth.layers_csc(17, 0, nl, n)
    bias = [np.full(n, 0.10 if l != die else -100.0, np.float32) for l in range(nl)]
    layers = [(cp[l], ri, v, bias[l]) for l in range(nl)]
    log(f"few-tile tail dies m={m}")
    gpu, o, cats = run_both(n, layers, y0)
    assert cats.size == 0
    counts = oracle.padded_live_counts(o, nl)
    assert counts[die] == m and counts[die + 1] == 0
    kinds, _ = gpu.net.layer_info()
    ran = [l for l in range(nl) if sdnn_kind(kinds[l]) != "none"]
    assert ran == list(range(len(ran)))
    assert sdnn_kind(kinds[5]) == "k_layer_gfm_small"
    # the host learns of the empty list a few layers after the device (6 layers of lead)
    assert die + 1 < len(ran) <= die + 12, len(ran)
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("kind", ["one-weight", "ell"])
def test_few_tile_rows_die_one_by_one(kind):
    """Rows that die at chosen layers: a dense row of value 1/4 - 2^-k / 4 under 32 weights of 1/16 and
    bias -1/4 drifts from the fixed point 1/4 by a doubling amount and dies near layer k, while rows
    of value 1/2 saturate and survive. The list shrinks a few rows per layer through the few-tile
    layers, with compactions as the host's bound drops. "ell": one weight per layer differs, so the
    layers go through the ELL instead of the 16-bit source lists."""
    n, nl, bias = 6000, 40, -0.25
    die = [1 + (7 * r) % 17 for r in range(42)]
    vals = [0.25 - 0.25 * 2.0 ** -k for k in die] + [0.5] * 6
    y0 = np.repeat(np.asarray(vals, np.float32)[:, None], n, axis=1)
    cp, ri, v = synth.layers_csc(18, 0, nl, n)
    if kind == "ell":
        v = v.copy()
        for l in range(nl):
            v[cp[l][0]] = np.float32(0.125)
    layers = [(cp[l], ri, v, np.full(n, bias, np.float32)) for l in range(nl)]
    log(f"few-tile rows die one by one kind={kind}")
    gpu, o, cats = run_both(n, layers, y0, equal_values=kind == "one-weight")
    counts = oracle.padded_live_counts(o, nl)
    assert counts[-1] >= 6 and any(8 < c <= 16 for c in counts) and any(c <= 8 for c in counts)
    kinds, _ = gpu.net.layer_info()
    assert sdnn_kind(kinds[nl - 1]) == "k_layer_gfm_small"
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("equal_values", [False, True])
@pytest.mark.parametrize("n,m", [(1024, 400), (4096, 200), (16384, 80), (65536, 30)])
def test_structured_networks(n, m, equal_values):
    """Structured (RadiX-Net style) layers: a radix-2 base DNN Kronecker-expanded by 16 x 16 blocks,
    randomly relabelled per copy of the D base layers (Fig. 1, Table 1). Inputs of mixed density so
    that some rows survive; two copies and a layer of the third, on both kernel paths."""
    d = synth.radix_depth(n)
    nl = 2 * d + 1
    bias = {1024: -0.30, 4096: -0.35, 16384: -0.40, 65536: -0.45}[n]
    side = int(round(n ** 0.5))
    y0 = synth.inputs(40 + d, side, 0, m, "mixed", 0.3, 0.8)
    cp, ri, v = synth.radix_layers_csc(21, 0, nl, n)
    layers = [(cp[l], ri, v, np.full(n, bias, np.float32)) for l in range(nl)]
    log(f"structured n={n} m={m} layers={nl} equal_values={equal_values}")
    gpu, o, cats = run_both(n, layers, y0, equal_values=equal_values)
    assert 0 < cats.size < m
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("order", ["one-by-one", "reversed", "mixed-bias"])
def test_structured_duplicate_columns(order):
    """In structured layers every 16 columns of a Kronecker block share their sources, weights and
    bias, so their outputs are equal: the library computes one column per group once the next
    layer's sources have been mapped to the representatives, which needs that layer loaded right
    after. "one-by-one": layers loaded one per call, in order; "reversed": one per call from the last
    layer back, so no layer's successor is mapped and every column is computed; "mixed-bias": one
    column's bias differs, so that layer is not uniform and keeps all its columns."""
    n, m = 16384, 80
    d = synth.radix_depth(n)
    nl = 2 * d + 1
    side = int(round(n ** 0.5))
    y0 = synth.inputs(40 + d, side, 0, m, "mixed", 0.3, 0.8)
    cp, ri, v = synth.radix_layers_csc(22, 0, nl, n)
    bias = [np.full(n, -0.40, np.float32) for _ in range(nl)]
    if order == "mixed-bias":
        bias[d][123] = np.float32(-0.41)
    layers = [(cp[l], ri, v, bias[l]) for l in range(nl)]
    gpu = GpuNet(n, nl, equal_values=True)  # one column per group needs the equal-value kernels
    seq = range(nl - 1, -1, -1) if order == "reversed" else range(nl)
    for l in seq:
        gpu.load(l, cp[l], ri, v, bias[l])
    log(f"structured duplicate columns order={order}")
    cats = gpu.run(y0)
    o = oracle.run(y0, layers, 32.0, threads=4)
    assert 0 < cats.size < m
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("n", [4096, 5001])
def test_maximum_column_degree(n):
    """A column may hold up to 4096 sources, and the ELL width is a layer's largest degree: one
    column of each layer takes 4096 sources, the others 0 to 8; signed weights, biases of both
    signs, on both kernel paths (LDS tiles at 4096, global tiles at 5001)."""
    rng = np.random.default_rng(n)
    nl, m = 3, 40
    layers = []
    for _ in range(nl):
        deg = rng.integers(0, 9, size=n)
        deg[rng.integers(n)] = 4096
        cp, ri, v = synth.random_csc(rng, n, deg, -1.0, 1.0)
        layers.append((cp, ri, v, rng.uniform(-0.3, 0.3, size=n).astype(np.float32)))
    y0 = (rng.random((m, n)) < 0.5).astype(np.float32) * rng.uniform(0, 2, (m, n)).astype(np.float32)
    log(f"maximum column degree n={n} m={m}")
    gpu, o, cats = run_both(n, layers, y0)
    assert gpu.net.kernel_path == (0 if n <= 4096 else 1)
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("equal_values", [False, True])
@pytest.mark.parametrize("n,m", [(4096, 900), (2048, 1800), (1024, 3000)])
def test_fused_tile_heights(n, m, equal_values):
    """Rows that stay live (Bernoulli(0.6) inputs) reach the launch that runs every remaining layer
    once two layers have kept 90% of them, with tiles of 4, 8 or 16 rows per workgroup for these
    widths and row counts; with equal_values each height reads its own grouped column order."""
    nl = 8
    rng = np.random.default_rng(n + m)
    y0 = (rng.random((m, n)) < 0.6).astype(np.float32)
    cp, ri, v = synth.layers_csc(14, 0, nl, n)
    layers = [(cp[l], ri, v, np.full(n, -0.35, np.float32)) for l in range(nl)]
    log(f"fused tile heights n={n} m={m} layers={nl} equal_values={equal_values}")
    gpu, o, cats = run_both(n, layers, y0, equal_values=equal_values)
    kinds = [sdnn_kind(k) for k in gpu.net.layer_info()[0]]
    log(f"kinds {kinds}")
    assert kinds[-1] == "k_layers_lds" and cats.size == m
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("case", ["tiles", "counted", "last-fused"])
def test_structured_lds_columns(case):
    """Structured networks on widths staged in LDS: one column per group of equal columns in the
    one-layer LDS kernel, in layer 0 by counts (written as fp32 rows) and in the launch that runs
    every remaining layer; the final rows are expanded through the last layer's groups.
    "tiles": more live rows than the fused launch takes, so several layers run one by one;
    "counted": 2^24 binary inputs, layer 0 by counts; "last-fused": the fused launch ends the run."""
    n, m, nl, bias = {"tiles": (1024, 3000, 6, -0.30), "counted": (4096, 4200, 4, -0.35),
                      "last-fused": (1024, 600, 21, -0.30)}[case]
    d = synth.radix_depth(n)
    side = int(round(n ** 0.5))
    y0 = synth.inputs(50 + d, side, 0, m, "mixed", 0.05, 0.35)
    cp, ri, v = synth.radix_layers_csc(24, 0, nl, n)
    layers = [(cp[l], ri, v, np.full(n, bias, np.float32)) for l in range(nl)]
    log(f"structured LDS columns case={case} n={n} m={m} layers={nl}")
    gpu, o, cats = run_both(n, layers, y0, equal_values=True)
    kinds = [sdnn_kind(k) for k in gpu.net.layer_info()[0]]
    log(f"kinds {kinds}")
    if case == "tiles":
        assert kinds[1] == "k_layer_lds"
    if case == "counted":
        assert kinds[0] == "k_pack_bits+k_layer_count"
    if case == "last-fused":
        assert kinds[-1] == "k_layers_lds"
    assert 0 < cats.size < m
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("n,ell", [(40000, False), (40001, True), (6000, False)])
def test_two_byte_codes(n, ell):
    """Layer inputs of 257 to 4096 distinct values are gathered as two-byte codes where the fp32
    tiles are larger than an XCD's L2 (40,000 neurons: 5 MB; at 6000 the same layers gather fp32).
    Weights that are multiples of 1/64 on binary inputs give layer 0 a few hundred output values:
    its one-byte codes overflow (it writes fp32), and the rows with two nonzero inputs (15%) die, so
    layer 1's inputs come through the repack: its one-byte codes overflow, and the two-byte encoding
    of the repacked tiles holds.
    Layer 1's random weights give millions of values: both encodings of layer 2's inputs overflow
    (fp32 gather). Layer 2 saturates every entry (one value: one-byte codes for layer 3); layer 3's
    weights, multiples of 1/2048 on inputs of 32, give a few hundred values again, so layer 4
    gathers two-byte codes after the one-byte success re-enabled them; layer 5 reads fp32 (one
    value per column, n in all). With ell, layers 1 and 4 have columns of up to 40 sources (the ELL
    form of the kernels), on a width that is not a multiple of 32."""
    m = 2600
    rng = np.random.default_rng(57 + ell + n)

    def layer(l, step, k, bias, scale=0.125):
        cp, ri, _ = synth.layers_csc(60 + ell, l, 1, n, k=k)
        if step:
            v = (rng.integers(1, 65, size=ri.size) * np.float32(step)).astype(np.float32)
        else:
            v = rng.uniform(0.0, scale, size=ri.size).astype(np.float32)
        return cp[0], ri, v, np.full(n, bias, np.float32)

    wide = 40 if ell else 32
    layers = [layer(0, 1 / 64, 32, -1.2), layer(1, 0, wide, -0.2), layer(2, 1 / 64, 32, 40.0),
              layer(3, 1 / 2048, 32, -0.3), layer(4, 0, wide, -0.2, 0.05), layer(5, 1 / 64, 32, -0.3)]
    y0 = (rng.random((m, n)) < 0.5).astype(np.float32)
    for i in np.nonzero(rng.random(m) < 0.15)[0]:
        y0[i] = 0.0
        y0[i, rng.choice(n, 2, replace=False)] = 1.0
    log(f"two-byte codes n={n} ell={ell}")
    gpu, o, cats = run_both(n, layers, y0)
    kind, launches = gpu.net.layer_info()
    names = [sdnn_kind(k) for k in kind]
    log(f"kernels {names}, launches {launches.tolist()}")
    counts = gpu.net.live_counts()
    assert counts[0] == m and 2048 <= counts[1] < 0.9 * m  # rows die in layer 0: its outputs are repacked
    coded = "k_layer_gfm_u16" if n * 32 * 4 > 4 << 20 else "k_layer_gfm"
    assert names == ["k_pack_bits+k_layer_bits", coded, "k_layer_gfm", "k_layer_gfm_u8", coded, "k_layer_gfm"]
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("n,nvals", [(6000, 256), (6000, 257), (40000, 4096), (40000, 4097)])
def test_dictionary_capacity(n, nvals):
    """The dictionaries' capacities, exactly: layer 0 gives column j the single source j with weight
    1 + (j mod (nvals - 1)) / 8192 (exact in fp32) and bias -0.5, so on binary rows its outputs take
    exactly nvals distinct values (+0 and nvals - 1 others). 256 values fit the one-byte codes that
    layer 0 writes and layer 1 gathers; at 257 layer 0 rewrites fp32 tiles. At 40,000 neurons (where
    two-byte codes are tried: the fp32 tiles outgrow the L2) 4096 values fit the two-byte codes of
    layer 1's inputs; 4097 overflow them and layer 1 gathers fp32 tiles. 2100 rows."""
    m = 2100
    rng = np.random.default_rng(71)
    cp0 = np.arange(n + 1, dtype=np.int64)
    ri0 = np.arange(n, dtype=np.int32)
    v0 = (1.0 + (np.arange(n) % (nvals - 1)) / 8192.0).astype(np.float32)
    layers = [(cp0, ri0, v0, np.full(n, -0.5, np.float32))]
    for l in (1, 2):
        cp, ri, _ = synth.layers_csc(70, l, 1, n)
        layers.append((cp[0], ri, rng.uniform(0.0, 0.125, size=ri.size).astype(np.float32),
                       np.full(n, -0.2, np.float32)))
    y0 = (rng.random((m, n)) < 0.5).astype(np.float32)
    log(f"dictionary capacity: n={n}, {nvals} values")
    gpu, o, cats = run_both(n, layers, y0)
    names = [sdnn_kind(k) for k in gpu.net.layer_info()[0]]
    log(f"kernels {names}")
    assert (gpu.net.live_counts() == m).all()
    expect = {256: ["k_pack_bits+k_layer_bits(codes)", "k_layer_gfm_u8"],
              257: ["k_pack_bits+k_layer_bits", "k_layer_gfm"],
              4096: ["k_pack_bits+k_layer_bits", "k_layer_gfm_u16"],
              4097: ["k_pack_bits+k_layer_bits", "k_layer_gfm"]}[nvals]
    assert names == expect + ["k_layer_gfm"]
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("nvals", [256, 257])
def test_repack_dictionary_capacity(nvals):
    """The repack that writes the next layer's one-byte codes, at the dictionary's exact bound.
    Layer 0 passes the binary inputs through (identity, weight 1, bias 0: two values, one-byte
    codes). Layer 1 gives column j < 3000 the single source j with weight 1 + (j mod (nvals - 1)) /
    8192 and bias -0.5, and kills the other columns (bias -5), so its outputs take exactly nvals
    values, and the 15% of rows whose ones all lie in the killed columns die. The repack after it
    writes layer 2's inputs as codes for 256 values; for 257 it falls back to fp32 tiles."""
    n, m = 6000, 2600
    rng = np.random.default_rng(73)
    cp0 = np.arange(n + 1, dtype=np.int64)
    ri0 = np.arange(n, dtype=np.int32)
    v1 = (1.0 + (np.arange(n) % (nvals - 1)) / 8192.0).astype(np.float32)
    b1 = np.where(np.arange(n) < n // 2, -0.5, -5.0).astype(np.float32)
    cp2, ri2, _ = synth.layers_csc(72, 2, 1, n)
    w2 = rng.uniform(0.0, 0.125, size=ri2.size).astype(np.float32)
    layers = [(cp0, ri0, np.ones(n, np.float32), np.zeros(n, np.float32)), (cp0, ri0, v1, b1),
              (cp2[0], ri2, w2, np.full(n, -0.2, np.float32))]
    y0 = (rng.random((m, n)) < 0.5).astype(np.float32)
    dying = rng.random(m) < 0.15
    y0[dying, : n // 2] = 0.0
    log(f"repack dictionary capacity: {nvals} values")
    gpu, o, cats = run_both(n, layers, y0)
    names = [sdnn_kind(k) for k in gpu.net.layer_info()[0]]
    counts = gpu.net.live_counts()
    log(f"kernels {names}, live counts {counts.tolist()}")
    assert counts[1] == m and 2048 <= counts[2] <= 0.9 * m
    assert names == ["k_pack_bits+k_layer_bits(codes)", "k_layer_gfm_u8",
                     "k_layer_gfm_u8" if nvals <= 256 else "k_layer_gfm"]
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("equal_values", [False, True])
@pytest.mark.parametrize("nl", [2, 5])
def test_structured_code_layer_columns(nl, equal_values):
    """A structured network on more than 256 rows: layer 0 writes one-byte codes (by counts with
    equal_values), layer 1 gathers them and, with equal_values and its successor's sources mapped to
    the representatives, computes one column per group of equal columns and stores all of their
    segments. nl=2: layer 1 is the last layer, whose final rows are expanded through its groups."""
    n, m = 8192, 700
    d = synth.radix_depth(n)
    rng = np.random.default_rng(nl)
    y0 = (rng.random((m, n)) < rng.uniform(0.1, 0.5, size=(m, 1))).astype(np.float32)
    cp, ri, v = synth.radix_layers_csc(23, 0, nl, n)
    layers = [(cp[l], ri, v, np.full(n, -0.40, np.float32)) for l in range(nl)]
    log(f"structured code layer columns n={n} nl={nl} (D={d}) equal_values={equal_values}")
    gpu, o, cats = run_both(n, layers, y0, equal_values=equal_values)
    kinds, _ = gpu.net.layer_info()
    assert sdnn_kind(kinds[1]) == "k_layer_gfm_u8"
    assert 0 < cats.size < m
    assert_parity(gpu, o, cats)


def test_profiling_modes():
    """Mode 1 times every layer that ran; mode 2 only the large ones (here: the layers entered with more
    than 256 live rows, on the global-tile path)."""
    n, m, nl, bias = 6000, 1100, 12, -0.40
    rng = np.random.default_rng(7)
    y0 = (rng.random((m, n)) < rng.uniform(0.10, 0.40, size=(m, 1))).astype(np.float32)
    cp, ri, v = synth.layers_csc(12, 0, nl, n)
    gpu = GpuNet(n, nl)
    gpu.load(0, cp, ri, v, np.full((nl, n), bias, np.float32))
    gpu.net.set_profiling(True)
    gpu.run(y0)
    ms, runs = gpu.net.layer_times()
    assert (runs == 1).all() and (ms > 0).all()
    gpu.net.set_profiling(True, large_only=True)
    gpu.run(y0)
    gpu.run(y0)
    ms, runs = gpu.net.layer_times()
    counts = gpu.net.live_counts()
    large = [l for l in range(nl) if l == 0 or counts[l] > 256]
    assert runs[large].tolist() == [2] * len(large) and (ms[large] > 0).all()
    assert (runs[[l for l in range(nl) if l not in large]] == 0).all()
    gpu.net.set_profiling(False)


@pytest.mark.parametrize("n,m", [(16384, 700), (65536, 400)])
@pytest.mark.parametrize("wkind", ["three-values", "random"])
def test_value_agnostic_large_binary_batch(n, m, wkind):
    """More than 256 binary rows through layers whose weights vary per edge and whose biases vary per
    neuron, at both bit-tile heights (32 rows up to 16384 neurons, 16 beyond). "three-values":
    weights drawn from {1/16, 3/32, 1/8} and biases from {-0.40, -0.45}, so layer 0's outputs take
    154 distinct values: layer 0 writes one-byte codes through the value dictionary (claiming slots
    with compare-and-swap across workgroups) and layer 1 gathers them with each edge's weight.
    "random": uniform random weights, so the dictionary overflows and layer 0 is computed again with
    fp32 outputs, which layer 1 gathers."""
    nl = 3
    rng = np.random.default_rng(n + (0 if wkind == "random" else 1))
    cp, ri, v = synth.layers_csc(31, 0, nl, n)
    layers = []
    for l in range(nl):
        if wkind == "random":
            w = rng.uniform(0.02, 0.2, size=v.size).astype(np.float32)
        else:
            w = rng.choice(np.array([1 / 16, 3 / 32, 1 / 8], np.float32), size=v.size).astype(np.float32)
        b = rng.choice(np.array([-0.40, -0.45], np.float32), size=n).astype(np.float32)
        layers.append((cp[l], ri, w, b))
    y0 = (rng.random((m, n)) < rng.uniform(0.15, 0.5, size=(m, 1))).astype(np.float32)
    y0[3] = 0.0
    log(f"value-agnostic large binary batch n={n} m={m} weights={wkind}")
    gpu, o, cats = run_both(n, layers, y0)
    kinds, launches = gpu.net.layer_info()
    if wkind == "random":
        assert sdnn_kind(kinds[0]) == "k_pack_bits+k_layer_bits" and launches[0] == 3
        assert sdnn_kind(kinds[1]) == "k_layer_gfm"
    else:
        assert sdnn_kind(kinds[0]) == "k_pack_bits+k_layer_bits(codes)"
        assert sdnn_kind(kinds[1]) == "k_layer_gfm_u8"
    assert oracle.padded_live_counts(o, nl)[1] > 256
    assert_parity(gpu, o, cats)


@pytest.mark.parametrize("n,kind", [(6000, "binary"), (6000, "scaled"), (12001, "binary"), (2048, "binary"),
                                    (2048, "scaled")])
def test_mixed_degrees_up_to_32(n, kind):
    """Layers whose largest column degree is 32 but whose columns hold 8 to 32 sources, with signed
    per-edge weights: the kernels that read 32 sources per column from 16-bit lists must pad the
    shorter columns with no-op terms. More than 256 rows, so the large-layer kernels run on the
    global-tile path (one-byte codes after a binary layer 0, fp32 tiles after a scaled one), and
    the per-layer and fused LDS kernels on widths staged in LDS."""
    rng = np.random.default_rng(n + len(kind))
    m, nl = 900, 5
    layers = []
    for _ in range(nl):
        deg = rng.integers(8, 33, size=n)
        deg[rng.integers(n)] = 32
        cp, ri, v = synth.random_csc(rng, n, deg, -0.05, 0.25)
        layers.append((cp, ri, v, rng.uniform(-0.35, -0.25, size=n).astype(np.float32)))
    y0 = (rng.random((m, n)) < rng.uniform(0.3, 0.7, size=(m, 1))).astype(np.float32)
    if kind == "scaled":
        y0 *= np.float32(1.25)
    log(f"mixed degrees up to 32 n={n} kind={kind}")
    gpu, o, cats = run_both(n, layers, y0)
    assert 0 < cats.size
    assert_parity(gpu, o, cats)
