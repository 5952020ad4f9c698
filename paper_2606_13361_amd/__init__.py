"""MI355X-native prefill and prefix-reuse continuation attention.

The product is libkvr.so (HIP kernels for gfx950 behind the C ABI in
include/kvr.h); ``kvr`` is its Python binding.
"""
from . import kvr  # noqa: F401
from .kvr import (KvrError, kvr_abi_version, kvr_cache_append, kvr_continue,  # noqa: F401
                  kvr_continue_batched, kvr_prefill, kvr_workspace_bytes, make_desc, workspace_for)
