"""ctypes binding of libsdnn.so (include/sdnn.h). Argument marshalling only: every step of the
inference runs in the library's HIP kernels. There is no fallback; a missing library is an error."""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(HERE, "libsdnn.so")
_lib = None

STATUS = {0: "SDNN_OK", 1: "SDNN_EINVAL", 2: "SDNN_ENOMEM", 3: "SDNN_EDEVICE", 4: "SDNN_ESTATE", 5: "SDNN_ERANGE"}
EXPORTED_SYMBOLS = [
    "sdnn_create", "sdnn_load_layers", "sdnn_workspace_bytes", "sdnn_infer", "sdnn_categories",
    "sdnn_live_counts", "sdnn_final_rows", "sdnn_destroy", "sdnn_last_error", "sdnn_kernel_path",
    "sdnn_set_profiling", "sdnn_layer_times", "sdnn_layer_info", "sdnn_enable_equal_value_kernels",
    "sdnn_infer_static",
]
KERNEL_KINDS = {0: "none", 1: "k_layer_lds", 2: "k_layer_gfm", 3: "k_layer_gfm_u8", 4: "k_layer_gfm_small",
                5: "k_pack_bits+k_layer_bits", 6: "k_pack_bits+k_layer_bits(codes)", 7: "k_pack_bits+k_layer_count",
                8: "k_layers_lds", 9: "k_layer_gfm_u16"}


class SdnnError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status
        self.name = STATUS.get(status, str(status))


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load the built libsdnn.so; raises if it has not been built (see __graft_entry__.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build the HIP library first (python -m paper_1909_05631_amd.build)")
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.sdnn_create.argtypes = [ctypes.POINTER(vp), i32, i32, ctypes.c_float]
        L.sdnn_load_layers.argtypes = [vp, i32, i32, vp, vp, vp, vp, vp]
        L.sdnn_workspace_bytes.argtypes = [vp, i64]
        L.sdnn_workspace_bytes.restype = sz
        L.sdnn_infer.argtypes = [vp, vp, i64, vp, sz, vp]
        L.sdnn_categories.argtypes = [vp, vp, i64, ctypes.POINTER(i64)]
        L.sdnn_live_counts.argtypes = [vp, vp]
        L.sdnn_final_rows.argtypes = [vp, vp, i64, vp]
        L.sdnn_destroy.argtypes = [vp]
        L.sdnn_destroy.restype = None
        L.sdnn_last_error.argtypes = []
        L.sdnn_last_error.restype = ctypes.c_char_p
        L.sdnn_kernel_path.argtypes = [vp]
        L.sdnn_kernel_path.restype = i32
        L.sdnn_set_profiling.argtypes = [vp, i32]
        L.sdnn_layer_times.argtypes = [vp, vp, vp]
        L.sdnn_layer_info.argtypes = [vp, vp, vp]
        L.sdnn_enable_equal_value_kernels.argtypes = [vp, i32]
        L.sdnn_infer_static.argtypes = [vp, vp, i64, vp]
        for name in ("sdnn_create", "sdnn_load_layers", "sdnn_infer", "sdnn_categories", "sdnn_live_counts",
                     "sdnn_final_rows", "sdnn_set_profiling", "sdnn_layer_times", "sdnn_layer_info",
                     "sdnn_enable_equal_value_kernels", "sdnn_infer_static"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise SdnnError(status, load_library().sdnn_last_error().decode())


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _dev_ptr(t) -> int:
    """Device address of a torch tensor (or an int address)."""
    return t if isinstance(t, int) else int(t.data_ptr())


def _stream_handle(stream) -> int | None:
    if stream is None:
        return None
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


class Net:
    """A network of `n_layers` layers of `n_neurons` neurons (one libsdnn handle).

    equal_value_kernels: opt in to the kernels that exploit layers whose weights and biases are all
    equal (sdnn_enable_equal_value_kernels); off by default."""

    def __init__(self, n_neurons: int, n_layers: int, ymax: float = 32.0, equal_value_kernels: bool = False):
        L = load_library()
        h = ctypes.c_void_p()
        _check(L.sdnn_create(ctypes.byref(h), n_neurons, n_layers, ymax))
        self._lib = L  # held so that close() still works while the interpreter shuts down
        self._h = h
        if equal_value_kernels:
            _check(L.sdnn_enable_equal_value_kernels(h, 1))
        self.n = n_neurons
        self.n_layers = n_layers
        self.ymax = ymax
        self.rows = 0

    def close(self):
        if getattr(self, "_h", None):
            self._lib.sdnn_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    @property
    def kernel_path(self) -> int:
        return int(load_library().sdnn_kernel_path(self._h))

    def load_layers(self, l0: int, col_ptr: np.ndarray, row_idx: np.ndarray, val: np.ndarray, bias: np.ndarray,
                    stream=None) -> None:
        """col_ptr (nl, n+1) or (n+1,) int64 CSC offsets into row_idx/val; bias (nl, n) or (n,)."""
        col_ptr = np.ascontiguousarray(col_ptr, dtype=np.int64).reshape(-1, self.n + 1)
        bias = np.ascontiguousarray(bias, dtype=np.float32).reshape(-1, self.n)
        row_idx = np.ascontiguousarray(row_idx, dtype=np.int32)
        val = np.ascontiguousarray(val, dtype=np.float32)
        nl = col_ptr.shape[0]
        if bias.shape[0] != nl:
            raise ValueError("bias and col_ptr disagree on the number of layers")
        if col_ptr.size and (col_ptr.max() > row_idx.size or col_ptr.max() > val.size):
            raise ValueError("col_ptr runs past row_idx/val")
        _check(load_library().sdnn_load_layers(self._h, l0, nl, _p(col_ptr), _p(row_idx), _p(val), _p(bias),
                                               _stream_handle(stream)))

    def workspace_bytes(self, n_rows: int) -> int:
        return int(load_library().sdnn_workspace_bytes(self._h, n_rows))

    def infer(self, y0, n_rows: int, workspace, workspace_bytes: int, stream=None) -> None:
        """y0 / workspace: device tensors (or raw device addresses)."""
        self.rows = n_rows
        _check(load_library().sdnn_infer(self._h, _dev_ptr(y0) if n_rows else None, n_rows, _dev_ptr(workspace),
                                         workspace_bytes, _stream_handle(stream)))

    def infer_static(self, y0, n_rows: int, stream=None) -> None:
        """sdnn_infer with the library's static device workspace (no allocation; see sdnn.h)."""
        self.rows = n_rows
        _check(load_library().sdnn_infer_static(self._h, _dev_ptr(y0) if n_rows else None, n_rows,
                                                _stream_handle(stream)))

    def categories(self) -> np.ndarray:
        L = load_library()
        cnt = ctypes.c_int64(0)
        st = L.sdnn_categories(self._h, None, 0, ctypes.byref(cnt))
        if st not in (0, 5):
            _check(st)
        ids = np.empty(max(cnt.value, 1), dtype=np.int64)
        _check(L.sdnn_categories(self._h, _p(ids), ids.size, ctypes.byref(cnt)))
        return ids[: cnt.value]

    def live_counts(self) -> np.ndarray:
        out = np.empty(self.n_layers + 1, dtype=np.int64)
        _check(load_library().sdnn_live_counts(self._h, _p(out)))
        return out

    def set_profiling(self, enable, large_only: bool = False) -> None:
        """Per-layer HIP-event timing of later runs: off, every layer, or large layers only."""
        _check(load_library().sdnn_set_profiling(self._h, 0 if not enable else (2 if large_only else 1)))

    def layer_info(self) -> tuple[np.ndarray, np.ndarray]:
        """Per layer of the last run: kernel family (KERNEL_KINDS) and number of launches."""
        kind = np.zeros(self.n_layers, dtype=np.int32)
        launches = np.zeros(self.n_layers, dtype=np.int32)
        _check(load_library().sdnn_layer_info(self._h, _p(kind), _p(launches)))
        return kind, launches

    def layer_times(self) -> tuple[np.ndarray, np.ndarray]:
        ms = np.zeros(self.n_layers, dtype=np.float64)
        runs = np.zeros(self.n_layers, dtype=np.int64)
        _check(load_library().sdnn_layer_times(self._h, _p(ms), _p(runs)))
        return ms, runs

    def final_rows(self, ids) -> np.ndarray:
        ids = np.ascontiguousarray(ids, dtype=np.int64)
        out = np.empty((ids.size, self.n), dtype=np.float32)
        _check(load_library().sdnn_final_rows(self._h, _p(ids), ids.size, _p(out)))
        return out
