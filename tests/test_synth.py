"""The seeded workload generator: structure of the weight layers and inputs (Sec. III, Sec. IV)."""
import numpy as np
import pytest

import synth


@pytest.mark.parametrize("n", [1024, 4096])
def test_layers_are_32_regular_without_duplicates(n):
    cp, ri, v = synth.layers_csc(3, 5, 3, n)
    k = 32
    assert cp.shape == (3, n + 1)
    for l in range(3):
        np.testing.assert_array_equal(cp[l], l * n * k + np.arange(n + 1) * k)
        cols = ri[l * n * k:(l + 1) * n * k].reshape(n, k)
        assert (np.diff(cols, axis=1) > 0).all()  # ascending, hence no duplicate (i, j)
        assert cols.min() >= 0 and cols.max() < n
        assert (np.bincount(cols.ravel(), minlength=n) == k).all()  # 32 per row as well
    assert (v == np.float32(1.0 / 16.0)).all()


def test_layers_are_unions_of_permutations():
    n = 1024
    perm = synth.layer_perms(2, 7, n)
    for a in range(32):
        assert np.array_equal(np.sort(perm[a]), np.arange(n))
    cp, ri, _ = synth.layers_csc(2, 7, 1, n)
    cols = ri.reshape(n, 32)
    edges = set()
    for a in range(32):
        edges.update(zip(range(n), perm[a].tolist()))
    assert len(edges) == 32 * n
    for j in range(0, n, 97):
        assert set(cols[j].tolist()) == {i for (i, jj) in edges if jj == j}


def test_generation_is_deterministic_and_layer_addressable():
    a = synth.layers_csc(4, 10, 2, 1024)
    b = synth.layers_csc(4, 10, 2, 1024, threads=1)
    c = synth.layers_csc(4, 11, 1, 1024)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    np.testing.assert_array_equal(a[1][1024 * 32:], c[1])  # layer 11 alone == second layer of the chunk
    assert not np.array_equal(a[1][:1024 * 32], c[1])


def test_input_sets_prefix_and_density():
    big = synth.inputs(1, 32, 0, 400)
    small = synth.inputs(1, 32, 0, 100)
    mid = synth.inputs(1, 32, 150, 50)
    np.testing.assert_array_equal(big[:100], small)
    np.testing.assert_array_equal(big[150:200], mid)
    assert set(np.unique(big)) <= {0.0, 1.0}
    d = big.mean(axis=1)
    assert 0.14 < d.mean() < 0.30 and d.min() >= 0.04 and d.max() <= 0.5
    bern = synth.inputs(2, 64, 0, 50, "bernoulli", 0.6)
    assert abs(bern.mean() - 0.6) < 0.01
    mixed = synth.inputs(3, 32, 0, 200, "mixed", 0.2, 0.5)
    dm = mixed.mean(axis=1)
    assert dm.min() > 0.15 and dm.max() < 0.55


def test_config_table_matches_tables_1_and_2():
    from tests.golden import load
    bias = {n: b for n, b in load("table1_bias.txt")}
    conns = {(l, n): c for l, n, c in load("table2_connections.txt")}
    for cfg in synth.CONFIGS:
        assert cfg.bias == bias[cfg.n_neurons]
        assert cfg.k == 32
        assert cfg.total_nnz == conns[(cfg.n_layers, cfg.n_neurons)]


@pytest.mark.parametrize("n", [64, 128, 1024])
def test_radix_layers_are_32_regular(n):
    """Structured layers (Fig. 1, Table 1): 32 ascending sources per column, each neuron feeding 32."""
    d = synth.radix_depth(n)
    nl = 2 * d + 1
    cp, ri, v = synth.radix_layers_csc(5, 0, nl, n)
    for l in range(nl):
        np.testing.assert_array_equal(cp[l], l * n * 32 + np.arange(n + 1) * 32)
        cols = ri[l * n * 32:(l + 1) * n * 32].reshape(n, 32)
        assert (np.diff(cols, axis=1) > 0).all() and cols.min() >= 0 and cols.max() < n
        assert (np.bincount(cols.ravel(), minlength=n) == 32).all()
    assert (v == np.float32(1.0 / 16.0)).all()
    assert [synth.radix_depth(x) for x in (1024, 4096, 16384, 65536)] == [6, 8, 10, 12]  # Table 1 radix sets
    assert synth.radix_depth(1000) == 0 and synth.radix_depth(16) == 0


@pytest.mark.parametrize("n", [64, 128, 256])
def test_radix_copies_have_equal_path_counts(n):
    """Within one copy of the D base layers every input neuron reaches every output neuron by the same
    number of paths (one base path, 16 choices at each of the D - 1 inner layers), the property the
    paper gives for RadiX-Net DNNs; and undoing a copy's relabelling leaves the Kronecker form with
    blocks of 16 x 16."""
    d = synth.radix_depth(n)
    cp, ri, _ = synth.radix_layers_csc(6, 0, 2 * d, n)
    dense = []
    for l in range(2 * d):
        a = np.zeros((n, n), dtype=np.int64)
        cols = ri[l * n * 32:(l + 1) * n * 32].reshape(n, 32)
        for j in range(n):
            a[cols[j], j] = 1  # W(source, target)
        dense.append(a)
    for c in range(2):
        prod = np.eye(n, dtype=np.int64)
        for l in range(c * d, (c + 1) * d):
            prod = prod @ dense[l]
        assert (prod == 16 ** (d - 1)).all(), (c, np.unique(prod))
        perm = synth.radix_perm(6, c, n)
        assert np.array_equal(np.sort(perm), np.arange(n))
        for l in range(c * d, (c + 1) * d):
            base = dense[l][np.ix_(perm, perm)]  # base(s, t) = W(P(s), P(t))
            blocks = base.reshape(n // 16, 16, n // 16, 16)
            assert (blocks.min(axis=(1, 3)) == blocks.max(axis=(1, 3))).all()  # 16 x 16 blocks
            node = blocks[:, 0, :, 0]
            assert (node.sum(axis=0) == 2).all() and (node.sum(axis=1) == 2).all()
    assert not np.array_equal(synth.radix_perm(6, 0, n), synth.radix_perm(6, 1, n))
