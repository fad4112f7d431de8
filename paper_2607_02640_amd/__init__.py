"""MI355X-native windowed-KV frame attention (Metronome, arXiv 2607.02640).

The attention path lives in libmtn.so (HIP for gfx950 behind the C ABI of
include/mtn.h); this package is its thin Python binding.
"""
from ._lib import (Pool, Admission, MtnError, load, hbm_copy, hbm_read, EXPORTS, LIB_PATH,  # noqa: F401
                   MTN_OK, MTN_ERR_INVALID_ARG, MTN_ERR_BAD_SESSION, MTN_ERR_CHUNK_TOO_LARGE,
                   MTN_ERR_NO_SESSION_SLOT, MTN_ERR_POOL_EXHAUSTED, MTN_ERR_SESSION_FULL,
                   MTN_ERR_DEVICE, MTN_ERR_BAD_STATE, MTN_ERR_UNSUPPORTED, MTN_ERR_HOST_MEMORY)
