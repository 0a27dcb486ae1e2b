"""MI355X-native phase-split decoder forward pass (prefill + KV-cache decode).

The compute lives in libll.so (hand-written gfx950 HIP kernels behind the C ABI declared in
include/ll.h and include/ll_ops.h); ``binding`` marshals arguments to it via ctypes.
"""
from .binding import LLError, Model, load_library, upload_weights  # noqa: F401
