"""NOVA-KV hot path for MI355X (gfx950): 2-bit VQ KV-cache encode and decode attention.

The compute lives in ``libnovakv.so`` (hand-written HIP, C ABI in
``include/nova_kv.h``); this package is its Python binding.
"""

from .api import (NOALLOC_SCRATCH_BYTES, Band, CacheLayout, NovaKVParams, append_decode_attn,  # noqa: F401
                  append_decode_attn_noalloc, band_shape, check_metadata, set_debug,
                  code_pool_shape, decode_attn, decode_workspace_bytes, encode, prepare_append_decode,
                  prepare_decode, prepare_encode, scale_pool_shape)
from ._native import NovaKVError  # noqa: F401
