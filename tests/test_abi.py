"""The C ABI without a GPU: the library loads, exports every entry point include/sdnn.h declares, and
rejects malformed arguments on the host before touching any device."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_1909_05631_amd import sdnn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "sdnn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sdnn_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(sdnn.library_path()):
        from paper_1909_05631_amd import build
        build.build()
    return sdnn.load_library()


def test_every_declared_symbol_is_exported(lib):
    names = declared_symbols()
    assert set(sdnn.EXPORTED_SYMBOLS) == set(names)
    for name in names:
        assert hasattr(lib, name), name


def test_kernel_kinds_match_the_header():
    """The binding's names of the layer kernel families cover exactly the values of the header's
    sdnn_kernel_kind enum (what sdnn_layer_info reports)."""
    text = open(os.path.join(ROOT, "include", "sdnn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    body = re.search(r"typedef enum \{(.*?)\} sdnn_kernel_kind;", text, flags=re.S).group(1)
    values = {int(v) for v in re.findall(r"SDNN_KERNEL_[A-Z0-9_]+\s*=\s*(\d+)", body)}
    assert values == set(sdnn.KERNEL_KINDS)


def _status(fn, *args):
    return fn(*args)


def test_create_validation(lib):
    h = ctypes.c_void_p()
    assert lib.sdnn_create(ctypes.byref(h), 0, 10, 32.0) == 1
    assert b"n_neurons" in lib.sdnn_last_error()
    assert lib.sdnn_create(ctypes.byref(h), 70000, 10, 32.0) == 1
    assert lib.sdnn_create(ctypes.byref(h), 16, 0, 32.0) == 1
    assert lib.sdnn_create(ctypes.byref(h), 16, 4, 0.0) == 1
    assert lib.sdnn_create(ctypes.byref(h), 16, 4, float("inf")) == 1
    assert lib.sdnn_create(ctypes.byref(h), 16, 4, float("nan")) == 1
    assert lib.sdnn_create(None, 16, 4, 32.0) == 1
    assert lib.sdnn_create(ctypes.byref(h), 16, 4, 32.0) == 0 and h.value
    lib.sdnn_destroy(h)
    lib.sdnn_destroy(None)


def test_kernel_path_by_width():
    assert sdnn.Net(1024, 1).kernel_path == 0
    assert sdnn.Net(4096, 1).kernel_path == 0
    assert sdnn.Net(16384, 1).kernel_path == 1
    assert sdnn.Net(65536, 1).kernel_path == 1


def _layer(n, rows_per_col):
    cp = np.zeros(n + 1, np.int64)
    cp[1:] = np.cumsum([len(r) for r in rows_per_col])
    ri = np.array([x for r in rows_per_col for x in r], np.int32)
    return cp, ri, np.ones(ri.size, np.float32)


@pytest.mark.parametrize("case,msg", [
    ("unsorted", "ascending"), ("duplicate", "ascending"), ("range", "out of range"), ("negative", "out of range"),
    ("nan_weight", "non-finite weight"), ("inf_bias", "non-finite bias"), ("decreasing", "decreasing"),
    ("layers", "outside"), ("gap", "does not start"),
])
def test_load_layers_rejects_malformed_csc(case, msg):
    n = 4
    net = sdnn.Net(n, 2)
    cp, ri, v = _layer(n, [[0, 2], [1], [], [0, 1, 3]])
    b = np.zeros(n, np.float32)
    l0, cps = 0, cp
    if case == "unsorted":
        ri[0], ri[1] = 2, 0
    elif case == "duplicate":
        ri[1] = 0
    elif case == "range":
        ri[2] = 4
    elif case == "negative":
        ri[2] = -1
    elif case == "nan_weight":
        v[3] = np.nan
    elif case == "inf_bias":
        b[1] = np.inf
    elif case == "decreasing":
        cps = cp.copy(); cps[2] = 0
    elif case == "layers":
        l0 = 2
    elif case == "gap":
        cps = np.stack([cp, cp])  # second layer must start at 6, not 0
        b = np.zeros((2, n), np.float32)
    with pytest.raises(sdnn.SdnnError) as ei:
        net.load_layers(l0, cps, ri, v, b)
    assert ei.value.name in ("SDNN_EINVAL",) and msg in str(ei.value)


def test_infer_before_load_is_a_state_error():
    net = sdnn.Net(8, 3)
    with pytest.raises(sdnn.SdnnError) as ei:
        net.infer(0, 0, 256, 1 << 20)
    assert ei.value.name == "SDNN_ESTATE"
    with pytest.raises(sdnn.SdnnError) as ei:
        net.categories()
    assert ei.value.name == "SDNN_ESTATE"


def test_workspace_bytes_grows_with_rows():
    net = sdnn.Net(1024, 3)
    a, b = net.workspace_bytes(0), net.workspace_bytes(1000)
    assert 0 < a < b
    assert b >= 2 * 1000 * 1024 * 4
    # the global-tile path keeps two buffers of 32-row tiles: 65 rows round up to 96
    assert sdnn.Net(65536, 2).workspace_bytes(65) >= 2 * 96 * 65536 * 4


def test_profiling_mode_out_of_range_is_einval():
    net = sdnn.Net(1024, 2)
    with pytest.raises(sdnn.SdnnError) as ei:
        _check = sdnn.load_library().sdnn_set_profiling(net._h, 3)
        sdnn._check(_check)
    assert ei.value.name == "SDNN_EINVAL"
