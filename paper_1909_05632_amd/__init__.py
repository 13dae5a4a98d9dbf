"""Frame-to-frame convolutional activation reuse on MI355X (gfx950).

The compute path is the HIP library ``libreuse_net.so`` (C ABI in
``include/reuse_net.h``); ``binding`` marshals arguments to it through ctypes
and uses torch only for device memory and streams.
"""
from .binding import (  # noqa: F401
    EXPORTS,
    LIB_PATH,
    RN_BF16,
    RN_F32,
    RN_HEAD_FULL,
    RN_HEAD_TILES,
    RN_U8,
    ReuseNet,
    ReuseNetError,
    load_library,
)
