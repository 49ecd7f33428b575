"""MI355X-native Sparse DNN Challenge inference (Kepner et al., 2019).

The computation runs in libsdnn.so (hand-written HIP for gfx950, C ABI declared in include/sdnn.h);
``paper_1909_05631_amd.sdnn`` is a thin ctypes binding with the same entry points. PyTorch is used
only for device memory and streams.
"""
from .sdnn import (  # noqa: F401
    Net, SdnnError, STATUS, load_library, library_path, EXPORTED_SYMBOLS,
)
