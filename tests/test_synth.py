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
