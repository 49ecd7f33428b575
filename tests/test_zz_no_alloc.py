"""sdnn_infer_static (the entry point for callers that cannot allocate) against sdnn_infer, through
the C ABI: two static runs in a row, the second on fewer rows, each equal to sdnn_infer's run on
the same input (categories, per-layer live counts, surviving rows); a batch too large for the static
workspace is refused before anything is enqueued."""
import numpy as np
import pytest

import synth
from tests.gpu_util import log, torch_cuda

pytestmark = pytest.mark.gpu

STATIC_BYTES = 64 << 20


def results(net, run, y0d, m):
    run(y0d, m)
    cats = net.categories()
    return cats, net.live_counts(), net.final_rows(cats)


@pytest.mark.parametrize("n,nl,m1,m2,bias", [(6000, 6, 700, 300, -0.40), (1024, 12, 2000, 900, -0.30)])
def test_static_workspace_matches_infer(n, nl, m1, m2, bias):
    from paper_1909_05631_amd import sdnn
    torch = torch_cuda()
    rng = np.random.default_rng(n)
    y0 = (rng.random((m1, n)) < rng.uniform(0.15, 0.5, size=(m1, 1))).astype(np.float32)
    cp, ri, v = synth.layers_csc(41, 0, nl, n)
    b = np.full((nl, n), bias, np.float32)
    ref, sta = sdnn.Net(n, nl), sdnn.Net(n, nl)
    for net in (ref, sta):
        net.load_layers(0, cp, ri, v, b)
    assert sta.workspace_bytes(m1) <= STATIC_BYTES
    stream = torch.cuda.current_stream()
    ya = torch.from_numpy(y0).cuda()
    yb = torch.from_numpy(np.ascontiguousarray(y0[:m2][::-1])).cuda()  # a different, smaller batch
    nb = ref.workspace_bytes(m1)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    want = [results(ref, lambda y, m: ref.infer(y, m, ws, nb, stream), y, m) for (y, m) in ((ya, m1), (yb, m2))]
    for i, (y, m) in enumerate(((ya, m1), (yb, m2))):
        log(f"static run {i}: n={n} rows={m}")
        got = results(sta, lambda y_, m_: sta.infer_static(y_, m_, stream), y, m)
        for g, w in zip(got, want[i]):
            np.testing.assert_array_equal(g, w)
        assert 0 < got[0].size < m


def test_static_workspace_refuses_large_batches():
    from paper_1909_05631_amd import sdnn
    torch = torch_cuda()
    n, nl = 6000, 2
    cp, ri, v = synth.layers_csc(41, 0, nl, n)
    net = sdnn.Net(n, nl)
    net.load_layers(0, cp, ri, v, np.full((nl, n), -0.4, np.float32))
    m = 3000
    assert net.workspace_bytes(m) > STATIC_BYTES
    y = torch.zeros((m, n), dtype=torch.float32, device="cuda")
    with pytest.raises(sdnn.SdnnError) as e:
        net.infer_static(y, m, torch.cuda.current_stream())
    assert e.value.name == "SDNN_ERANGE"
