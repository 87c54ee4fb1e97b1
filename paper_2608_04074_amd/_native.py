"""ctypes view of libnovakv.so (the C ABI declared in include/nova_kv.h).

Loading fails loudly when the library has not been built: there is no
fallback implementation of any call.
"""

from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libnovakv.so")

NOVA_KV_OK = 0
NOVA_KV_ERR_INVALID_ARG = 1
NOVA_KV_ERR_UNSUPPORTED = 2
NOVA_KV_ERR_WORKSPACE = 3
NOVA_KV_ERR_HIP = 4

NOVA_KV_F32 = 0
NOVA_KV_BF16 = 1

NOVA_KV_KEY_SCALE = 1  # nova_kv_params.flags: the key-scale format
NOVA_KV_FP8_CODEBOOKS = 2  # nova_kv_params.flags: codebooks stored as fp8 E4M3 bytes
NOVA_KV_SQ_VALUES = 4  # nova_kv_params.flags: the scalar (per-token affine INT2) value arm
NOVA_KV_BF16_TRANSFORMS = 8  # nova_kv_params.flags: t_k, t_k_inv_t and t_v stored as bf16

EXPORTED = (
    "nova_kv_encode",
    "nova_kv_decode_workspace_bytes",
    "nova_kv_decode_attn",
    "nova_kv_append_decode_attn",
    "nova_kv_append_decode_attn_noalloc",
    "nova_kv_check_metadata",
    "nova_kv_set_debug",
    "nova_kv_status_string",
    "nova_kv_last_error",
)


class Params(ctypes.Structure):
    _fields_ = [
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("group_dim", ctypes.c_int32),
        ("codebook_size", ctypes.c_int32),
        ("flags", ctypes.c_uint32),
        ("kbar", ctypes.c_void_p),
        ("t_k", ctypes.c_void_p),
        ("t_k_inv_t", ctypes.c_void_p),
        ("t_v", ctypes.c_void_p),
        ("cb_k", ctypes.c_void_p),
        ("cb_v", ctypes.c_void_p),
    ]


class Layout(ctypes.Structure):
    _fields_ = [
        ("block_size", ctypes.c_int32),
        ("blocks_per_seq", ctypes.c_int32),
        ("block_table", ctypes.c_void_p),
    ]


class Band(ctypes.Structure):
    _fields_ = [
        ("n_sink", ctypes.c_int32),
        ("n_rec", ctypes.c_int32),
        ("k", ctypes.c_void_p),
        ("v", ctypes.c_void_p),
    ]


NOVA_KV_MAX_BAND = 1024


class NovaKVError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"nova_kv status {status}: {detail}")
        self.status = status
        self.detail = detail


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m "
                               "paper_2608_04074_amd.build` (or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        L.nova_kv_encode.restype = ctypes.c_int
        # (params, layout, k, v, in_dtype, batch, n_new, start_pos, k_codes, v_codes,
        #  k_scales, v_sq, band, stream)
        L.nova_kv_encode.argtypes = [P(Params), P(Layout), vp, vp, ctypes.c_int, i32, i32, vp,
                                     vp, vp, vp, vp, P(Band), vp]
        L.nova_kv_decode_workspace_bytes.restype = ctypes.c_size_t
        L.nova_kv_decode_workspace_bytes.argtypes = [P(Params), i32, i32, i32]
        L.nova_kv_decode_attn.restype = ctypes.c_int
        # (params, layout, q, q_dtype, batch, num_q_heads, k_codes, v_codes, k_scales, v_sq,
        #  band, seq_lens, max_seq_len, window, sinks, softmax_scale, out, workspace, bytes, stream)
        L.nova_kv_decode_attn.argtypes = [P(Params), P(Layout), vp, ctypes.c_int, i32, i32, vp, vp, vp,
                                          vp, P(Band), vp, i32, i32, vp, ctypes.c_float, vp, vp,
                                          ctypes.c_size_t, vp]
        L.nova_kv_append_decode_attn.restype = ctypes.c_int
        # (params, layout, k_new, v_new, new_dtype, q, q_dtype, batch, num_q_heads, k_codes,
        #  v_codes, k_scales, v_sq, band, seq_lens, max_seq_len, window, sinks, softmax_scale,
        #  out, workspace, bytes, stream)
        L.nova_kv_append_decode_attn.argtypes = [P(Params), P(Layout), vp, vp, ctypes.c_int, vp,
                                                 ctypes.c_int, i32, i32, vp, vp, vp, vp, P(Band), vp,
                                                 i32, i32, vp, ctypes.c_float, vp, vp, ctypes.c_size_t, vp]
        L.nova_kv_append_decode_attn_noalloc.restype = ctypes.c_int
        # the arguments of nova_kv_append_decode_attn without (workspace, bytes)
        L.nova_kv_append_decode_attn_noalloc.argtypes = [P(Params), P(Layout), vp, vp, ctypes.c_int, vp,
                                                         ctypes.c_int, i32, i32, vp, vp, vp, vp, P(Band), vp,
                                                         i32, i32, vp, ctypes.c_float, vp, vp]
        L.nova_kv_check_metadata.restype = ctypes.c_int
        # (layout with a host block table, num_blocks, batch, seq_lens, max_seq_len, start_pos, n_new)
        L.nova_kv_check_metadata.argtypes = [P(Layout), i32, i32, vp, i32, vp, i32]
        L.nova_kv_set_debug.restype = None
        L.nova_kv_set_debug.argtypes = [i32, i32]
        L.nova_kv_status_string.restype = ctypes.c_char_p
        L.nova_kv_status_string.argtypes = [ctypes.c_int]
        L.nova_kv_last_error.restype = ctypes.c_char_p
        L.nova_kv_last_error.argtypes = []
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != NOVA_KV_OK:
        raise NovaKVError(status, lib().nova_kv_last_error().decode())
