"""Pins for the CPU oracle: each test ties it to something other than its own code.

- integer-valued networks, where fp32 is exact in any order, against a float64 dense product
  (the Sec. V loop written with a library matmul);
- random float networks against exact rational arithmetic, within the error bound of a fused
  multiply-add chain;
- hand-derived IEEE cases that fix the summation order, the fused multiply-add and the sign of zero;
- the closed form of an all-ones row through 32 weights of 1/16 per column;
- special cases that reduce to array indexing (one permutation per layer);
- invariants of the recurrence.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth


def dense_w(n, col_ptr, row_idx, val, dtype=np.float64):
    W = np.zeros((n, n), dtype=dtype)
    for j in range(n):
        for e in range(col_ptr[j], col_ptr[j + 1]):
            W[row_idx[e], j] = val[e]
    return W


def matlab_layer(Y, W, b, ymax):
    """Sec. V serial loop, one layer: the product, the bias on its nonzero entries, the clamp to [0, YMAX]."""
    Z = Y @ W
    Yn = Z + (Z != 0) * b[None, :]
    Yn[Yn < 0] = 0
    Yn[Yn > ymax] = ymax
    return Yn


def random_int_net(rng, n, nl, max_deg, wmax=3, bmax=4):
    layers = []
    for _ in range(nl):
        deg = rng.integers(0, max_deg + 1, size=n)
        cp, ri, _ = synth.random_csc(rng, n, deg)
        v = rng.integers(1, wmax + 1, size=ri.size) * rng.choice([-1, 1], size=ri.size)
        b = rng.integers(-bmax, bmax + 1, size=n).astype(np.float32)
        layers.append((cp, ri, v.astype(np.float32), b))
    return layers


@pytest.mark.parametrize("seed", range(12))
def test_integer_networks_match_float64_dense(seed):
    """All values are small integers, so fp32 is exact whatever the order: the oracle must equal the
    float64 dense evaluation of the Sec. V loop exactly, layer by layer, including live counts and
    categories. Catches transposed W, wrong indices, dropped terms, sign errors and the bias rule."""
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 40))
    m = int(rng.integers(1, 24))
    nl = int(rng.integers(1, 7))
    ymax = float(rng.choice([7.0, 20.0, 50.0]))
    layers = random_int_net(rng, n, nl, max_deg=min(n, 12))
    lo = -2 if seed % 3 == 0 else 0
    y0 = rng.integers(lo, 4, size=(m, n)).astype(np.float32)
    y0[rng.random(m) < 0.2] = 0  # some all-zero input rows
    o = oracle.Oracle(y0, ymax)
    Y = y0.astype(np.float64)
    counts = [int((np.abs(Y).sum(axis=1) > 0).sum())]
    for (cp, ri, v, b) in layers:
        o.layer(cp, ri, v, b)
        Y = matlab_layer(Y, dense_w(n, cp, ri, v), b.astype(np.float64), ymax)
        counts.append(int((Y.sum(axis=1) > 0).sum()))
        np.testing.assert_array_equal(o.rows(np.arange(m)), Y.astype(np.float32))
    np.testing.assert_array_equal(o.live_counts(), counts)
    np.testing.assert_array_equal(o.categories(), np.nonzero((Y > 0).any(axis=1))[0])


def test_bias_only_where_z_nonzero():
    """Sec. V adds b only where Z != 0 (a numeric nonzero mask); with b > 0 a column whose products cancel to
    exactly 0 must stay 0, while the Sec. II row-replication reading would give b."""
    n = 3
    # column 0: sources 0, 1 with weights 1, -1 -> z = y0 - y1 = 0 for y0 == y1
    # column 1: no sources -> z = 0 ; column 2: source 2 with weight 1
    cp = np.array([0, 2, 2, 3], dtype=np.int64)
    ri = np.array([0, 1, 2], dtype=np.int32)
    v = np.array([1.0, -1.0, 1.0], dtype=np.float32)
    b = np.array([5.0, 5.0, 0.25], dtype=np.float32)
    o = oracle.Oracle(np.array([[2.0, 2.0, 1.0]], dtype=np.float32), 32.0)
    o.layer(cp, ri, v, b)
    np.testing.assert_array_equal(o.rows([0])[0], np.array([0.0, 0.0, 1.25], dtype=np.float32))


def _single_column_case(y_src, w):
    n = len(y_src) + 1
    cp = np.zeros(n + 1, dtype=np.int64)
    cp[1:] = len(y_src)  # column 0 holds every source 0..n-2 in ascending order
    ri = np.arange(len(y_src), dtype=np.int32)
    v = np.asarray(w, dtype=np.float32)
    y0 = np.zeros((1, n), dtype=np.float32)
    y0[0, : len(y_src)] = y_src
    o = oracle.Oracle(y0, 1e30)
    o.layer(cp, ri, v, np.zeros(n, dtype=np.float32))
    return o.rows([0])[0, 0]


def test_summation_is_ascending_source_order():
    """IEEE round-to-nearest-even, worked by hand: 1 + 2^-24 rounds back to 1 (a tie to the even
    significand) but 2^-24 + 2^-24 = 2^-23 and 1 + 2^-23 is exact. So sources [1, 2^-24, 2^-24]
    sum to exactly 1 in ascending order, while [2^-24, 2^-24, 1] give 1 + 2^-23."""
    t = np.float32(2.0 ** -24)
    assert _single_column_case([1.0, t, t], [1, 1, 1]) == np.float32(1.0)
    assert _single_column_case([t, t, 1.0], [1, 1, 1]) == np.float32(1.0 + 2.0 ** -23)


def test_each_term_is_one_fused_multiply_add():
    """(1 + 2^-12)^2 = 1 + 2^-11 + 2^-24 exactly. Added to -(1 + 2^-11) with one rounding this is
    2^-24; rounding the product first (a tie, to even: 1 + 2^-11) would give 0."""
    a = 1.0 + 2.0 ** -12
    got = _single_column_case([1.0, a], [-(1.0 + 2.0 ** -11), a])
    assert got == np.float32(2.0 ** -24)


def test_cancellation_gives_positive_zero():
    got = _single_column_case([3.0, 3.0], [1.0, -1.0])
    assert got == 0.0 and not np.signbit(got)


@pytest.mark.parametrize("seed", range(6))
def test_random_float_networks_within_fma_chain_bound(seed):
    """Random real weights, one layer at a time from the oracle's own previous Y: the exact sum
    (Python Fractions) and the oracle's output must agree within gamma_n * sum|terms| for n fused
    multiply-adds (unit roundoff u = 2^-24), plus one rounding of the bias add."""
    rng = np.random.default_rng(77 + seed)
    n, m, nl, ymax = 16, 6, 4, 32.0
    u = Fraction(1, 2 ** 24)
    y0 = (rng.random((m, n)) < 0.6).astype(np.float32) * rng.uniform(0.0, 2.0, (m, n)).astype(np.float32)
    o = oracle.Oracle(y0, ymax)
    Y = y0.copy()
    for _ in range(nl):
        deg = rng.integers(0, 9, size=n)
        cp, ri, v = synth.random_csc(rng, n, deg, -1.0, 1.0)
        b = rng.uniform(-0.5, 0.5, size=n).astype(np.float32)
        o.layer(cp, ri, v, b)
        Yn = o.rows(np.arange(m))
        for i in range(m):
            if not (Y[i] != 0).any():
                assert (Yn[i] == 0).all()
                continue
            for j in range(n):
                terms = [Fraction(float(Y[i, ri[e]])) * Fraction(float(v[e]))
                         for e in range(cp[j], cp[j + 1]) if Y[i, ri[e]] != 0]
                z = sum(terms, Fraction(0))
                k = len(terms)
                tol = (k * u / (1 - k * u)) * sum(abs(t) for t in terms) if k else Fraction(0)
                t_exact = z + Fraction(float(b[j]))
                got = Fraction(float(Yn[i, j]))
                slack = tol + u * (abs(t_exact) + tol) + Fraction(1, 2 ** 140)
                if got == 0:
                    assert abs(z) <= tol or t_exact <= slack
                elif got == Fraction(ymax):
                    assert t_exact >= Fraction(ymax) - slack
                else:
                    assert z != 0 or tol > 0
                    assert abs(got - t_exact) <= slack
        Y = Yn


@pytest.mark.parametrize("bias", [-0.30, -0.35, -0.40, -0.45])
def test_closed_form_all_ones_row(bias):
    """With 32 weights of 1/16 in every column, an all-ones row gives y_{l+1} = min(32, max(0, 2 y_l + b)),
    i.e. y_l = min(32, 2^l (1 + b) - b): 1.7, 3.1, 5.9, 11.5, 22.7, 32 for b = -0.30. Every entry of the
    row equals the closed form to fp32 accuracy, and is exactly 32 from layer 6 on."""
    n, nl = 1024, 10
    cp, ri, v = synth.layers_csc(1, 0, nl, n)
    o = oracle.Oracle(np.ones((1, n), dtype=np.float32), 32.0)
    b = np.full(n, bias, dtype=np.float32)
    for l in range(nl):
        o.layer(cp[l], ri, v, b)
        row = o.rows([0])[0]
        exact = min(32.0, 2.0 ** (l + 1) * (1.0 + bias) - bias)
        assert np.all(row == row[0])
        if exact == 32.0:
            assert row[0] == np.float32(32.0)
        else:
            assert abs(float(row[0]) - exact) <= 2e-6 * exact


@pytest.mark.parametrize("bias", [-0.30, -0.35, -0.40, -0.45])
def test_tie_probe_constant_row(bias):
    """A constant row c = fp32(-b)/2 makes 2c + b = 0 exactly. The oracle's sequential fp32 sum of the
    32 products c/16 (exact, a power-of-two scaling) must equal numpy's sequential cumulative sum,
    and the result then decides whether the row survives layer 1 -- a test that detects any other
    summation order at the granularity of whole rows."""
    n = 1024
    c = np.float32(-np.float32(bias)) / np.float32(2.0)
    cp, ri, v = synth.layers_csc(1, 0, 2, n)
    o = oracle.Oracle(np.full((1, n), c, dtype=np.float32), 32.0)
    b = np.full(n, bias, dtype=np.float32)
    o.layer(cp[0], ri, v, b)
    seq = np.cumsum(np.full(32, c * np.float32(1.0 / 16.0), dtype=np.float32), dtype=np.float32)[-1]
    t = np.float32(seq + np.float32(bias))
    expect = t if t > 0 else np.float32(0.0)
    row = o.rows([0])[0]
    assert np.all(row == expect)
    assert 2 * Fraction(float(c)) + Fraction(float(np.float32(bias))) == 0  # exact value of z + b
    if bias == -0.30:
        # the sequential sum lands just above -b: the row lives through layer 1, then dies
        assert t > 0
        o.layer(cp[1], ri, v, b)
        np.testing.assert_array_equal(o.live_counts(), [1, 1, 0])


@pytest.mark.parametrize("bias", [0.0, -0.25])
def test_single_permutation_layers_are_column_shuffles(bias):
    """One weight of 1 per column: W(i, s(i)) = 1 moves column i to column s(i), so
    Y_{l+1} = clip(Y_l[:, s^-1] + b * (Y_l[:, s^-1] != 0), 0, YMAX) with numpy indexing and one fp32 add."""
    rng = np.random.default_rng(5)
    n, m, ymax = 50, 9, 32.0
    y = rng.uniform(0, 3, (m, n)).astype(np.float32) * (rng.random((m, n)) < 0.7)
    o = oracle.Oracle(y, ymax)
    for l in range(5):
        s = rng.permutation(n)
        inv = np.argsort(s)
        cp = np.arange(n + 1, dtype=np.int64)
        ri = inv.astype(np.int32)  # column j's single source is s^-1(j)
        v = np.ones(n, dtype=np.float32)
        b = np.full(n, bias, dtype=np.float32)
        o.layer(cp, ri, v, b)
        z = y[:, inv]
        y = np.where(z != 0, z + np.float32(bias), np.float32(0)).astype(np.float32)
        y = np.clip(y, 0, ymax).astype(np.float32)
        np.testing.assert_array_equal(o.rows(np.arange(m)), y)


def test_identity_layers_leave_y_unchanged():
    rng = np.random.default_rng(9)
    n, m = 33, 7
    y = rng.uniform(0, 31, (m, n)).astype(np.float32) * (rng.random((m, n)) < 0.5)
    o = oracle.Oracle(y, 32.0)
    cp = np.arange(n + 1, dtype=np.int64)
    for _ in range(3):
        o.layer(cp, np.arange(n, dtype=np.int32), np.ones(n, np.float32), np.zeros(n, np.float32))
    np.testing.assert_array_equal(o.rows(np.arange(m)), y)


def test_invariants_on_config_network():
    """0 <= Y <= YMAX; the live count never grows; a dead row stays dead; permuting the input rows
    permutes every output bit for bit."""
    n, nl, m = 1024, 16, 96
    y0 = synth.inputs(7, 32, 0, m, "mixed", 0.15, 0.55)
    cp, ri, v = synth.layers_csc(1, 0, nl, n)
    b = np.full(n, -0.30, dtype=np.float32)
    perm = np.random.default_rng(3).permutation(m)
    o, op = oracle.Oracle(y0), oracle.Oracle(y0[perm])
    alive = np.ones(m, dtype=bool)
    for l in range(nl):
        o.layer(cp[l], ri, v, b)
        op.layer(cp[l], ri, v, b)
        Y = o.rows(np.arange(m))
        assert Y.min() >= 0 and Y.max() <= 32
        now = (Y > 0).any(axis=1)
        assert not (now & ~alive).any()
        alive = now
        np.testing.assert_array_equal(op.rows(np.arange(m)), Y[perm])
    c = o.live_counts()
    assert (np.diff(c) <= 0).all()
    assert 0 < c[-1] < m  # the mixed set straddles the survival threshold
    np.testing.assert_array_equal(np.sort(perm[op.categories()]), o.categories())


def test_float64_matlab_semantics_agree_on_robust_rows():
    """The paper's listing runs in double. On the config network, fp32 and float64 must give the same
    categories for every row whose smallest |z + b| stays well away from 0, and close values."""
    n, nl, m = 1024, 12, 64
    y0 = synth.inputs(8, 32, 0, m, "mixed", 0.2, 0.5)
    cp, ri, v = synth.layers_csc(1, 0, nl, n)
    b = np.full(n, -0.30, dtype=np.float32)
    o = oracle.Oracle(y0)
    Y = y0.astype(np.float64)
    for l in range(nl):
        o.layer(cp[l], ri, v, b)
        Y = matlab_layer(Y, dense_w(n, cp[l], ri, v), b.astype(np.float64), 32.0)
    _, per_row = o.margin()
    robust = per_row > 1e-3
    assert robust.sum() >= m // 2
    cat32 = np.zeros(m, dtype=bool)
    cat32[o.categories()] = True
    cat64 = (Y > 0).any(axis=1)
    np.testing.assert_array_equal(cat32[robust], cat64[robust])
    Y32 = o.rows(np.arange(m))
    np.testing.assert_allclose(Y32[robust], Y[robust], rtol=1e-3, atol=1e-4)


def test_empty_and_degenerate_batches():
    o = oracle.Oracle(np.zeros((0, 5), dtype=np.float32))
    cp = np.array([0, 1, 1, 2, 2, 2], dtype=np.int64)
    o.layer(cp, np.array([1, 0], np.int32), np.array([1, 1], np.float32), np.zeros(5, np.float32))
    assert o.categories().size == 0 and list(o.live_counts()) == [0, 0]
    o1 = oracle.Oracle(np.array([[2.0]], dtype=np.float32), 3.0)  # one neuron, clamped at YMAX
    o1.layer(np.array([0, 1], np.int64), np.array([0], np.int32), np.array([4.0], np.float32), np.zeros(1, np.float32))
    np.testing.assert_array_equal(o1.rows([0]), [[3.0]])
    with pytest.raises(ValueError):
        oracle.Oracle(np.ones((2, 2), np.float32), 0.0)
    with pytest.raises(ValueError):
        o1.layer(np.array([0, 1], np.int64), np.array([5], np.int32), np.array([1.0], np.float32), np.zeros(1, np.float32))


def test_threads_do_not_change_results():
    n, nl, m = 1024, 6, 40
    y0 = synth.inputs(9, 32, 0, m, "mixed", 0.2, 0.5)
    cp, ri, v = synth.layers_csc(1, 0, nl, n)
    b = np.full(n, -0.30, dtype=np.float32)
    o1, o4 = oracle.Oracle(y0), oracle.Oracle(y0)
    for l in range(nl):
        o1.layer(cp[l], ri, v, b, threads=1)
        o4.layer(cp[l], ri, v, b, threads=4)
    np.testing.assert_array_equal(o1.rows(np.arange(m)), o4.rows(np.arange(m)))
    np.testing.assert_array_equal(o1.live_counts(), o4.live_counts())


# ---- the margin and the smallest final row maximum (diagnostics of the oracle)

def exact_margins(y0, layers, ymax):
    """Integer networks, evaluated exactly in float64: per row, min |z + b| over every layer and
    every entry with z != 0 (inf if none), the same with |z| in place of |z + b|, and the last
    layer's minimum alone; plus the final Y."""
    Y = y0.astype(np.float64)
    n = y0.shape[1]
    best = np.full(y0.shape[0], np.inf)
    best_z = np.full(y0.shape[0], np.inf)
    last = np.full(y0.shape[0], np.inf)
    for (cp, ri, v, b) in layers:
        Z = Y @ dense_w(n, cp, ri, v)
        nz = Z != 0
        T = Z + b.astype(np.float64)[None, :]
        last = np.where(nz, np.abs(T), np.inf).min(axis=1) if n else last
        best = np.minimum(best, last)
        best_z = np.minimum(best_z, np.where(nz, np.abs(Z), np.inf).min(axis=1))
        Y = np.clip(np.where(nz, T, 0.0), 0.0, ymax)
    return best, best_z, last, Y


@pytest.mark.parametrize("seed", range(8))
def test_margin_on_integer_networks_is_exact(seed):
    """Every value is a small integer, so |z + b| is exact: the oracle's per-row margins must equal
    the float64 evaluation exactly. Across the seeds the margin differs from the minimum of |z| and
    from the last layer's minimum on many rows, so tracking |z|, or restarting at every layer, fails."""
    rng = np.random.default_rng(3000 + seed)
    n, m, nl, ymax = int(rng.integers(4, 30)), int(rng.integers(8, 30)), int(rng.integers(2, 6)), 40.0
    layers = random_int_net(rng, n, nl, max_deg=min(n, 8))
    y0 = rng.integers(0, 3, size=(m, n)).astype(np.float32)
    o = oracle.Oracle(y0, ymax)
    for layer in layers:
        o.layer(*layer)
    best, best_z, last, Y = exact_margins(y0, layers, ymax)
    m_all, per_row = o.margin()
    np.testing.assert_array_equal(per_row, best)
    assert m_all == best.min()
    differs_z = int((best_z != best).sum())
    differs_last = int((last != best).sum())
    assert differs_z > 0 or differs_last > 0 or not np.isfinite(best).any()
    cats = (Y > 0).any(axis=1)
    expect = Y[cats].max(axis=1).min() if cats.any() else np.inf
    assert o.min_final_rowmax() == expect


def test_margin_planted_mistakes_are_caught():
    """The integer-network check above, summed over its seeds, sees rows where |z| and |z + b| have
    different minima and rows whose minimum is reached before the last layer: a margin computed
    from |z| or restarted per layer cannot pass it."""
    diff_z = diff_last = 0
    for seed in range(8):
        rng = np.random.default_rng(3000 + seed)
        n, m, nl = int(rng.integers(4, 30)), int(rng.integers(8, 30)), int(rng.integers(2, 6))
        layers = random_int_net(rng, n, nl, max_deg=min(n, 8))
        y0 = rng.integers(0, 3, size=(m, n)).astype(np.float32)
        best, best_z, last, _ = exact_margins(y0, layers, 40.0)
        diff_z += int((best_z != best).sum())
        diff_last += int((last != best).sum())
    assert diff_z > 10 and diff_last > 10


def test_margin_single_column_by_hand():
    """Column 0 sums 1 * 0.5 + 1 * 0.25 = 0.75 and adds b = -0.5: |z + b| = 0.25 (|z| would be 0.75).
    Column 1 has no source, so z = 0 and its bias -0.1 is not applied: it must not count (it would
    give 0.1). Column 2 sums 1 * 2 = 2, b = -4: clamped to 0, |z + b| = 2."""
    n = 3
    cp = np.array([0, 2, 2, 3], dtype=np.int64)
    ri = np.array([0, 1, 0], dtype=np.int32)
    v = np.array([0.5, 0.25, 2.0], dtype=np.float32)
    b = np.array([-0.5, -0.1, -4.0], dtype=np.float32)
    o = oracle.Oracle(np.array([[1.0, 1.0, 0.0], [0.0, 0.0, 5.0]], dtype=np.float32), 32.0)
    o.layer(cp, ri, v, b)
    m, per_row = o.margin()
    assert m == 0.25
    np.testing.assert_array_equal(per_row, [0.25, np.inf])  # row 1 feeds no column: no term at all
    np.testing.assert_array_equal(o.rows([0, 1]), [[0.25, 0.0, 0.0], [0.0, 0.0, 0.0]])
    assert o.min_final_rowmax() == 0.25


def test_margin_tie_probe_by_hand():
    """The tie probe at b = -0.30: a constant row c = fp32(0.3)/2 = 5033165 * 2^-25 on the
    configs' network (32 weights of 1/16 per column). Each product c/16 = 5033165 * 2^-29 is exact;
    the exact sum of 32 of them is 2c = fp32(0.3), so z + b would be 0, but the sequential fp32
    sum (recomputed here with numpy float32 scalars, round to nearest even) ends 3 * 2^-25 above
    it: every entry of layer 1 has |z + b| = 3 * 2^-25 = 8.94e-8. Layer 2 then sums 32 terms of
    (3 * 2^-25)/16 = 6 * 2^-25 exactly and adds b: |z + b| is about 0.3, so the margin stays at
    layer 1's value (a per-layer restart would report 0.3), and the row dies."""
    n = 1024
    c = np.float32(0.3) / np.float32(2.0)
    assert Fraction(float(c)) == Fraction(5033165, 2 ** 25)
    acc = np.float32(0.0)
    for _ in range(32):
        acc = np.float32(acc + np.float32(c * np.float32(1.0 / 16.0)))
    t1 = np.float32(acc + np.float32(-0.30))
    assert Fraction(float(t1)) == Fraction(3, 2 ** 25)
    cp, ri, v = synth.layers_csc(1, 0, 2, n)
    b = np.full(n, -0.30, dtype=np.float32)
    o = oracle.Oracle(np.full((1, n), c, dtype=np.float32), 32.0)
    o.layer(cp[0], ri, v, b)
    assert o.margin()[0] == float(t1)
    assert o.min_final_rowmax() == float(t1)
    o.layer(cp[1], ri, v, b)
    assert o.margin()[0] == float(t1)
    assert o.live == 0 and o.min_final_rowmax() == np.inf


@pytest.mark.parametrize("bias", [-0.30, -0.45])
def test_min_final_rowmax_closed_form(bias):
    """An all-ones row saturates at YMAX = 32 from layer 6 on (closed form y_l = min(32, 2^l (1 + b) - b)),
    so after 8 layers its row maximum is exactly 32, while an all-zero row is never a category."""
    n = 1024
    cp, ri, v = synth.layers_csc(1, 0, 8, n)
    y0 = np.zeros((2, n), dtype=np.float32)
    y0[1] = 1.0
    o = oracle.Oracle(y0, 32.0)
    for l in range(8):
        o.layer(cp[l], ri, v, np.full(n, bias, dtype=np.float32))
    np.testing.assert_array_equal(o.categories(), [1])
    assert o.min_final_rowmax() == 32.0
