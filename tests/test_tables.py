"""The paper's tables: connection counts (Table 2) and the rate metric (Table 3)."""
import pytest

from tests.golden import load


def test_table2_is_32_times_layers_times_neurons():
    rows = load("table2_connections.txt")
    assert len(rows) == 12
    for layers, neurons, conns in rows:
        assert conns == 32 * layers * neurons


def test_table3_rate_is_inputs_times_edges_over_time():
    """Rate = (# inputs) x (# connections) / time with 60,000 inputs. The printed rates are the
    arithmetic truncated to three figures, except the 65536 x 480 row, which prints 299e6 where the
    arithmetic gives 298.4e6."""
    import math
    for neurons, layers, conns, secs, rate in load("table3_timing.txt"):
        assert conns == 32 * layers * neurons
        r = 60000 * conns / secs / 1e6
        if (neurons, layers) == (65536, 480):
            assert abs(r - rate) < 1.0
        else:
            assert math.floor(r) == rate, (neurons, layers, r)
