"""Python binding of the NOVA-KV C ABI: marshals torch device tensors into the calls.

Every step of the hot path runs in the HIP kernels of libnovakv.so; this module
only checks dtypes/shapes/devices, hands over raw device pointers and the
current HIP stream, and raises on a non-OK status.
"""

from __future__ import annotations

import contextlib
import ctypes
from typing import Optional

import torch

from . import _native as nat

__all__ = ["NovaKVParams", "CacheLayout", "Band", "band_shape", "encode", "decode_attn", "append_decode_attn",
           "append_decode_attn_noalloc", "NOALLOC_SCRATCH_BYTES", "check_metadata", "set_debug",
           "decode_workspace_bytes", "code_pool_shape", "scale_pool_shape", "prepare_encode",
           "prepare_decode", "prepare_append_decode"]


def _stream_ptr(stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _on_stream(stream: Optional[torch.cuda.Stream]):
    """Context in which temporaries of a call are created: the call's stream.

    The output and the zero-filled workspace that a call allocates for itself
    are then created and filled on the stream the kernels run on, so the
    fill is ordered before the launch, and the caching allocator only hands
    their memory to later work of that same stream once they are freed."""
    return torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()


def _require(t: torch.Tensor, name: str, dtypes, numel: Optional[int] = None) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")


class NovaKVParams:
    """Per-layer calibration outputs resident on the device (see nova_kv_params).

    ``key_scale`` selects the key-scale format (one bf16 scale per cached key;
    the key codebooks are then trained on normalized coefficients), and every
    call then takes a ``k_scales`` pool of shape ``scale_pool_shape``.
    Codebooks are fp16, or fp8 E4M3 bytes given as uint8 tensors (both sides
    in the same format).  ``sq_values`` selects the scalar value arm (values
    as per-token affine INT2 in the rotation t_v; cb_v unused, may be None),
    and every call then takes a ``v_sq`` pool of shape ``sq_pool_shape``.
    The transforms t_k, t_k_inv_t and t_v are fp32, or all three bf16 (the
    paper's serving storage of the bases), read as exactly those values.
    """

    def __init__(self, kbar, t_k, t_k_inv_t, t_v, cb_k, cb_v, group_dim: int = 4,
                 codebook_size: int = 256, key_scale: bool = False, sq_values: bool = False):
        hkv, d = kbar.shape
        L = d // group_dim
        _require(kbar, "kbar", (torch.float32,), hkv * d)
        for name, t in (("t_k", t_k), ("t_k_inv_t", t_k_inv_t), ("t_v", t_v)):
            _require(t, name, (torch.float32, torch.bfloat16), hkv * d * d)
        if not t_k.dtype == t_k_inv_t.dtype == t_v.dtype:
            raise TypeError("t_k, t_k_inv_t and t_v must have the same storage (fp32, or bf16)")
        self.bf16_transforms = t_k.dtype == torch.bfloat16
        self.sq_values = bool(sq_values)
        if self.sq_values and cb_v is None:
            cb_v = cb_k  # unused by the scalar value arm
        for name, t in (("cb_k", cb_k), ("cb_v", cb_v)):
            _require(t, name, (torch.float16, torch.uint8), hkv * L * codebook_size * group_dim)
        if cb_k.dtype != cb_v.dtype:
            raise TypeError("cb_k and cb_v must have the same format (fp16, or fp8 E4M3 as uint8)")
        self.fp8_codebooks = cb_k.dtype == torch.uint8
        self.num_kv_heads, self.head_dim = hkv, d
        self.group_dim, self.codebook_size = group_dim, codebook_size
        self.kbar, self.t_k, self.t_k_inv_t, self.t_v = kbar, t_k, t_k_inv_t, t_v
        self.cb_k, self.cb_v = cb_k, cb_v
        self.key_scale = bool(key_scale)
        flags = (nat.NOVA_KV_KEY_SCALE if self.key_scale else 0) | \
            (nat.NOVA_KV_FP8_CODEBOOKS if self.fp8_codebooks else 0) | \
            (nat.NOVA_KV_SQ_VALUES if self.sq_values else 0) | \
            (nat.NOVA_KV_BF16_TRANSFORMS if self.bf16_transforms else 0)
        self._c = nat.Params(hkv, d, group_dim, codebook_size, flags, kbar.data_ptr(), t_k.data_ptr(),
                             t_k_inv_t.data_ptr(), t_v.data_ptr(), cb_k.data_ptr(),
                             cb_v.data_ptr())

    @property
    def groups(self) -> int:
        return self.head_dim // self.group_dim

    @classmethod
    def from_arrays(cls, arrays: dict, device="cuda", key_scale: bool = False,
                    sq_values: bool = False, bf16_transforms: bool = False) -> "NovaKVParams":
        """From host arrays: kbar/t_k/t_k_inv_t/t_v float32, cb_k/cb_v float16, or uint8
        fp8 E4M3 codes ([Hkv][...]).  bf16_transforms: t_k, t_k_inv_t and t_v are
        stored as bf16 (rounded to nearest even from fp32)."""
        tdt = torch.bfloat16 if bf16_transforms else torch.float32
        f32 = {k: torch.as_tensor(arrays[k]).to(torch.float32).to(torch.float32 if k == "kbar" else tdt)
               .contiguous().to(device) for k in ("kbar", "t_k", "t_k_inv_t", "t_v")}
        f16 = {"cb_v": None}
        for k in ("cb_k", "cb_v"):
            if arrays.get(k) is None:
                continue
            t = torch.as_tensor(arrays[k])
            f16[k] = (t if t.dtype == torch.uint8 else t.to(torch.float16)).contiguous().to(device)
        return cls(**f32, **f16, key_scale=key_scale, sq_values=sq_values)

    @property
    def c(self) -> nat.Params:
        return self._c


class CacheLayout:
    """Code-pool layout (see nova_kv_layout); ``block_table`` is a device int32 [B][blocks_per_seq]."""

    def __init__(self, block_size: int, blocks_per_seq: int = 1,
                 block_table: Optional[torch.Tensor] = None):
        if block_table is not None:
            _require(block_table, "block_table", (torch.int32,))
        self.block_size, self.blocks_per_seq, self.block_table = block_size, blocks_per_seq, block_table
        self._c = nat.Layout(block_size, blocks_per_seq,
                             block_table.data_ptr() if block_table is not None else None)

    @classmethod
    def contiguous(cls, capacity: int) -> "CacheLayout":
        return cls(capacity, 1, None)

    @property
    def capacity(self) -> int:
        return self.block_size * self.blocks_per_seq

    @property
    def c(self) -> nat.Layout:
        return self._c


def code_pool_shape(params: NovaKVParams, layout: CacheLayout, batch: int, num_blocks=None):
    """Shape of one code pool: [num_blocks][Hkv][block_size][L]."""
    nb = batch * layout.blocks_per_seq if num_blocks is None else num_blocks
    return (nb, params.num_kv_heads, layout.block_size, params.groups)


def scale_pool_shape(params: NovaKVParams, layout: CacheLayout, batch: int, num_blocks=None):
    """Shape of the key-scale pool: [num_blocks][Hkv][block_size] (bf16 bit patterns)."""
    return code_pool_shape(params, layout, batch, num_blocks)[:3]


_SCALE_DTYPES = (torch.bfloat16, torch.int16, torch.uint16)


def _scales_ptr(params: NovaKVParams, k_scales: Optional[torch.Tensor], k_codes: torch.Tensor):
    """Device pointer of the key-scale pool (None outside the key-scale format)."""
    if not params.key_scale:
        return None
    if k_scales is None:
        raise ValueError("the key-scale format needs a k_scales pool")
    _require(k_scales, "k_scales", _SCALE_DTYPES, k_codes.numel() // params.groups)
    return k_scales.data_ptr()


def sq_pool_shape(params: NovaKVParams, layout: CacheLayout, batch: int, num_blocks=None):
    """Shape of the scalar value arm's pool: [num_blocks][Hkv][block_size][2] (scale, offset bf16 bits)."""
    return code_pool_shape(params, layout, batch, num_blocks)[:3] + (2,)


def _sq_ptr(params: NovaKVParams, v_sq: Optional[torch.Tensor], k_codes: torch.Tensor):
    """Device pointer of the (scale, offset) pool (None outside the scalar value arm)."""
    if not params.sq_values:
        return None
    if v_sq is None:
        raise ValueError("the scalar value arm needs a v_sq pool")
    _require(v_sq, "v_sq", _SCALE_DTYPES, 2 * (k_codes.numel() // params.groups))
    return v_sq.data_ptr()


def band_shape(params: NovaKVParams, batch: int, n_sink: int, n_rec: int):
    """Shape of each sink-plus-recent band buffer: [B][Hkv][n_sink + n_rec][D]."""
    return (batch, params.num_kv_heads, n_sink + n_rec, params.head_dim)


class Band:
    """Sink-plus-recent band (see nova_kv_band): the first n_sink and the last
    n_rec positions of every sequence held in bf16 in ``k`` and ``v``
    ([B][Hkv][n_sink + n_rec][D], bfloat16 or 16-bit integer bit patterns);
    position p sits in slot p < n_sink, else n_sink + p % n_rec."""

    def __init__(self, n_sink: int, n_rec: int, k: torch.Tensor, v: torch.Tensor):
        if n_sink < 0 or n_rec < 0 or not 1 <= n_sink + n_rec <= nat.NOVA_KV_MAX_BAND:
            raise ValueError(f"band sizes ({n_sink}, {n_rec}) outside 1 .. {nat.NOVA_KV_MAX_BAND} positions")
        _require(k, "band k", _SCALE_DTYPES)
        _require(v, "band v", (k.dtype,), k.numel())
        if k.dim() != 4 or k.shape[2] != n_sink + n_rec:
            raise ValueError("band buffers must be [B][Hkv][n_sink + n_rec][D]")
        self.n_sink, self.n_rec, self.k, self.v = n_sink, n_rec, k, v
        self._c = nat.Band(n_sink, n_rec, k.data_ptr(), v.data_ptr())

    def check(self, params: NovaKVParams, batch: int) -> None:
        if tuple(self.k.shape) != band_shape(params, batch, self.n_sink, self.n_rec):
            raise ValueError(f"band buffers of shape {tuple(self.k.shape)}, expected "
                             f"{band_shape(params, batch, self.n_sink, self.n_rec)}")

    @property
    def c(self) -> nat.Band:
        return self._c


def _band_ref(band: Optional[Band], params: NovaKVParams, batch: int):
    if band is None:
        return None
    band.check(params, batch)
    return ctypes.byref(band.c)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return nat.NOVA_KV_F32
    if t.dtype == torch.bfloat16:
        return nat.NOVA_KV_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def encode(params: NovaKVParams, layout: CacheLayout, k: torch.Tensor, v: torch.Tensor,
           start_pos: torch.Tensor, k_codes: torch.Tensor, v_codes: torch.Tensor,
           stream: Optional[torch.cuda.Stream] = None, k_scales: Optional[torch.Tensor] = None,
           band: Optional[Band] = None, v_sq: Optional[torch.Tensor] = None) -> None:
    """nova_kv_encode: k, v [B][n_new][Hkv][D] (fp32 or bf16), start_pos int32 [B]."""
    if k.dim() != 4:
        raise ValueError("k must be [B][n_new][Hkv][D]")
    b, n_new, hkv, d = k.shape
    if hkv != params.num_kv_heads or d != params.head_dim:
        raise ValueError("k does not match the parameters' head count / head_dim")
    _require(k, "k", (torch.float32, torch.bfloat16))
    _require(v, "v", (k.dtype,), k.numel())
    _require(start_pos, "start_pos", (torch.int32,), b)
    _require(k_codes, "k_codes", (torch.uint8,))
    _require(v_codes, "v_codes", (torch.uint8,), k_codes.numel())
    ks = _scales_ptr(params, k_scales, k_codes)
    nat.check(nat.lib().nova_kv_encode(
        ctypes.byref(params.c), ctypes.byref(layout.c), k.data_ptr(), v.data_ptr(), _dtype_code(k),
        b, n_new, start_pos.data_ptr(), k_codes.data_ptr(), v_codes.data_ptr(), ks,
        _sq_ptr(params, v_sq, k_codes), _band_ref(band, params, b), _stream_ptr(stream)))


def decode_workspace_bytes(params: NovaKVParams, batch: int, num_q_heads: int,
                           max_seq_len: int) -> int:
    return int(nat.lib().nova_kv_decode_workspace_bytes(ctypes.byref(params.c), batch,
                                                        num_q_heads, max_seq_len))


def decode_attn(params: NovaKVParams, layout: CacheLayout, q: torch.Tensor,
                k_codes: torch.Tensor, v_codes: torch.Tensor, seq_lens: torch.Tensor,
                max_seq_len: int, window: int = 0, sinks: Optional[torch.Tensor] = None,
                softmax_scale: float = 0.0, out: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None,
                stream: Optional[torch.cuda.Stream] = None,
                k_scales: Optional[torch.Tensor] = None, band: Optional[Band] = None,
                v_sq: Optional[torch.Tensor] = None) -> torch.Tensor:
    """nova_kv_decode_attn: q [B][Hq][D] (fp32 or bf16) -> out [B][Hq][D] fp32.

    A caller-provided workspace must be zero-filled before its first use; each
    call leaves it ready for the next.  When omitted, a zeroed one is allocated.
    """
    if q.dim() != 3 or q.shape[2] != params.head_dim:
        raise ValueError("q must be [B][Hq][D]")
    b, hq, d = q.shape
    _require(q, "q", (torch.float32, torch.bfloat16))
    _require(k_codes, "k_codes", (torch.uint8,))
    _require(v_codes, "v_codes", (torch.uint8,), k_codes.numel())
    _require(seq_lens, "seq_lens", (torch.int32,), b)
    if sinks is not None:
        _require(sinks, "sinks", (torch.float32,), hq)
    need = decode_workspace_bytes(params, b, hq, max_seq_len) if b > 0 else 0
    with _on_stream(stream):
        if out is None:
            out = torch.empty((b, hq, d), dtype=torch.float32, device=q.device)
        if workspace is None:
            workspace = torch.zeros(max(need, 1), dtype=torch.uint8, device=q.device)
    _require(out, "out", (torch.float32,), b * hq * d)
    _require(workspace, "workspace", (torch.uint8,))
    ks = _scales_ptr(params, k_scales, k_codes)
    nat.check(nat.lib().nova_kv_decode_attn(
        ctypes.byref(params.c), ctypes.byref(layout.c), q.data_ptr(), _dtype_code(q), b, hq,
        k_codes.data_ptr(), v_codes.data_ptr(), ks, _sq_ptr(params, v_sq, k_codes), _band_ref(band, params, b),
        seq_lens.data_ptr(),
        max_seq_len, window,
        sinks.data_ptr() if sinks is not None else None, float(softmax_scale), out.data_ptr(),
        workspace.data_ptr(), workspace.numel(), _stream_ptr(stream)))
    return out


def _append_decode_args(params, layout, k_new, v_new, q, k_codes, v_codes, seq_lens, max_seq_len, out,
                        workspace, window, sinks, softmax_scale, stream, k_scales, band, v_sq=None):
    if q.dim() != 3 or q.shape[2] != params.head_dim:
        raise ValueError("q must be [B][Hq][D]")
    b, hq, d = q.shape
    if tuple(k_new.shape) != (b, params.num_kv_heads, d):
        raise ValueError("k_new must be [B][Hkv][D]")
    _require(k_new, "k_new", (torch.float32, torch.bfloat16))
    _require(v_new, "v_new", (k_new.dtype,), k_new.numel())
    _require(q, "q", (torch.float32, torch.bfloat16))
    _require(k_codes, "k_codes", (torch.uint8,))
    _require(v_codes, "v_codes", (torch.uint8,), k_codes.numel())
    _require(seq_lens, "seq_lens", (torch.int32,), b)
    if sinks is not None:
        _require(sinks, "sinks", (torch.float32,), hq)
    _require(out, "out", (torch.float32,), b * hq * d)
    if workspace is not None:
        _require(workspace, "workspace", (torch.uint8,))
    ks = _scales_ptr(params, k_scales, k_codes)
    vp = ctypes.c_void_p
    return (ctypes.byref(params.c), ctypes.byref(layout.c), vp(k_new.data_ptr()), vp(v_new.data_ptr()),
            ctypes.c_int(_dtype_code(k_new)), vp(q.data_ptr()), ctypes.c_int(_dtype_code(q)),
            ctypes.c_int32(b), ctypes.c_int32(hq), vp(k_codes.data_ptr()), vp(v_codes.data_ptr()),
            vp(ks), vp(_sq_ptr(params, v_sq, k_codes)), _band_ref(band, params, b), vp(seq_lens.data_ptr()),
            ctypes.c_int32(max_seq_len),
            ctypes.c_int32(window),
            vp(sinks.data_ptr() if sinks is not None else None), ctypes.c_float(softmax_scale),
            vp(out.data_ptr()), vp(workspace.data_ptr() if workspace is not None else None),
            ctypes.c_size_t(workspace.numel() if workspace is not None else 0), vp(_stream_ptr(stream)))


def append_decode_attn(params: NovaKVParams, layout: CacheLayout, k_new: torch.Tensor, v_new: torch.Tensor,
                       q: torch.Tensor, k_codes: torch.Tensor, v_codes: torch.Tensor,
                       seq_lens: torch.Tensor, max_seq_len: int, window: int = 0,
                       sinks: Optional[torch.Tensor] = None, softmax_scale: float = 0.0,
                       out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                       stream: Optional[torch.cuda.Stream] = None,
                       k_scales: Optional[torch.Tensor] = None, band: Optional[Band] = None,
                       v_sq: Optional[torch.Tensor] = None) -> torch.Tensor:
    """nova_kv_append_decode_attn: store the step's k_new, v_new [B][Hkv][D] at
    position seq_lens[b] - 1 of the pools, then decode q [B][Hq][D] over the
    cache including them -> out [B][Hq][D] fp32.  Workspace as in decode_attn."""
    b, hq, d = q.shape
    need = decode_workspace_bytes(params, b, hq, max_seq_len) if b > 0 else 0
    with _on_stream(stream):
        if out is None:
            out = torch.empty((b, hq, d), dtype=torch.float32, device=q.device)
        if workspace is None:
            workspace = torch.zeros(max(need, 1), dtype=torch.uint8, device=q.device)
    args = _append_decode_args(params, layout, k_new, v_new, q, k_codes, v_codes, seq_lens, max_seq_len, out,
                               workspace, window, sinks, softmax_scale, stream, k_scales, band, v_sq)
    nat.check(nat.lib().nova_kv_append_decode_attn(*args))
    return out


def check_metadata(block_size: int, blocks_per_seq: int, block_table=None, num_blocks: int = 0,
                   seq_lens=None, max_seq_len: int = 0, start_pos=None, n_new: int = 0) -> None:
    """nova_kv_check_metadata on host arrays (numpy or CPU tensors, int32):
    raises NovaKVError naming the first offending entry."""
    import numpy as np

    def host(x):
        return None if x is None else np.ascontiguousarray(np.asarray(x, dtype=np.int32))

    bt, sl, sp = host(block_table), host(seq_lens), host(start_pos)
    batch = len(sl) if sl is not None else (len(sp) if sp is not None else 0)
    for name, x in (("seq_lens", sl), ("start_pos", sp)):
        if x is not None and len(x) != batch:
            raise ValueError(f"{name} must have one entry per sequence")
    if bt is not None and bt.size < batch * blocks_per_seq:
        raise ValueError("block_table must be [batch][blocks_per_seq]")
    ptr = lambda x: None if x is None else x.ctypes.data  # noqa: E731
    lay = nat.Layout(block_size, blocks_per_seq, ptr(bt))
    nat.check(nat.lib().nova_kv_check_metadata(ctypes.byref(lay), num_blocks, batch, ptr(sl), max_seq_len,
                                               ptr(sp), n_new))


def set_debug(on: bool, num_blocks: int = 0) -> None:
    """nova_kv_set_debug: entry points check their metadata on the host before
    launching (synchronizing; num_blocks <= 0: unknown pool size)."""
    nat.lib().nova_kv_set_debug(1 if on else 0, num_blocks)


NOALLOC_SCRATCH_BYTES = 32 << 20


def append_decode_attn_noalloc(params: NovaKVParams, layout: CacheLayout, k_new: torch.Tensor,
                               v_new: torch.Tensor, q: torch.Tensor, k_codes: torch.Tensor, v_codes: torch.Tensor,
                               seq_lens: torch.Tensor, max_seq_len: int, out: torch.Tensor, window: int = 0,
                               sinks: Optional[torch.Tensor] = None, softmax_scale: float = 0.0,
                               stream: Optional[torch.cuda.Stream] = None,
                               k_scales: Optional[torch.Tensor] = None, band: Optional[Band] = None,
                               v_sq: Optional[torch.Tensor] = None) -> torch.Tensor:
    """nova_kv_append_decode_attn_noalloc: the step of append_decode_attn with
    the library's fixed per-GPU scratch (NOALLOC_SCRATCH_BYTES) instead of a
    workspace; out is required, nothing is allocated.  Calls that overlap on
    one GPU race."""
    args = _append_decode_args(params, layout, k_new, v_new, q, k_codes, v_codes, seq_lens, max_seq_len, out,
                               None, window, sinks, softmax_scale, stream, k_scales, band, v_sq)
    # the same arguments without (workspace, bytes)
    nat.check(nat.lib().nova_kv_append_decode_attn_noalloc(*(args[:20] + args[22:])))
    return out


class PreparedCall:
    """One C call with every argument already marshalled: calling it costs a
    single foreign call, for loops that issue the same call many times (the
    tensors it was prepared from must stay alive and unchanged in place)."""

    def __init__(self, fn, args, keep):
        self._fn, self._args, self._keep = fn, args, keep

    def __call__(self) -> None:
        nat.check(self._fn(*self._args))


def prepare_encode(params: NovaKVParams, layout: CacheLayout, k: torch.Tensor, v: torch.Tensor,
                   start_pos: torch.Tensor, k_codes: torch.Tensor, v_codes: torch.Tensor,
                   stream: Optional[torch.cuda.Stream] = None,
                   k_scales: Optional[torch.Tensor] = None, band: Optional[Band] = None,
                   v_sq: Optional[torch.Tensor] = None) -> PreparedCall:
    """nova_kv_encode with the arguments of encode(), marshalled once."""
    if k.dim() != 4:
        raise ValueError("k must be [B][n_new][Hkv][D]")
    b, n_new, hkv, d = k.shape
    if hkv != params.num_kv_heads or d != params.head_dim:
        raise ValueError("k does not match the parameters' head count / head_dim")
    _require(k, "k", (torch.float32, torch.bfloat16))
    _require(v, "v", (k.dtype,), k.numel())
    _require(start_pos, "start_pos", (torch.int32,), b)
    _require(k_codes, "k_codes", (torch.uint8,))
    _require(v_codes, "v_codes", (torch.uint8,), k_codes.numel())
    ks = _scales_ptr(params, k_scales, k_codes)
    vp = ctypes.c_void_p
    args = (ctypes.byref(params.c), ctypes.byref(layout.c), vp(k.data_ptr()), vp(v.data_ptr()),
            ctypes.c_int(_dtype_code(k)), ctypes.c_int32(b), ctypes.c_int32(n_new),
            vp(start_pos.data_ptr()), vp(k_codes.data_ptr()), vp(v_codes.data_ptr()), vp(ks),
            vp(_sq_ptr(params, v_sq, k_codes)), _band_ref(band, params, b), vp(_stream_ptr(stream)))
    return PreparedCall(nat.lib().nova_kv_encode, args,
                        (params, layout, k, v, start_pos, k_codes, v_codes, k_scales, band, v_sq))


def prepare_decode(params: NovaKVParams, layout: CacheLayout, q: torch.Tensor,
                   k_codes: torch.Tensor, v_codes: torch.Tensor, seq_lens: torch.Tensor,
                   max_seq_len: int, out: torch.Tensor, workspace: torch.Tensor, window: int = 0,
                   sinks: Optional[torch.Tensor] = None, softmax_scale: float = 0.0,
                   stream: Optional[torch.cuda.Stream] = None,
                   k_scales: Optional[torch.Tensor] = None, band: Optional[Band] = None,
                   v_sq: Optional[torch.Tensor] = None) -> PreparedCall:
    """nova_kv_decode_attn with the arguments of decode_attn(), marshalled once
    (out and a zero-filled workspace are required here)."""
    if q.dim() != 3 or q.shape[2] != params.head_dim:
        raise ValueError("q must be [B][Hq][D]")
    b, hq, d = q.shape
    _require(q, "q", (torch.float32, torch.bfloat16))
    _require(k_codes, "k_codes", (torch.uint8,))
    _require(v_codes, "v_codes", (torch.uint8,), k_codes.numel())
    _require(seq_lens, "seq_lens", (torch.int32,), b)
    if sinks is not None:
        _require(sinks, "sinks", (torch.float32,), hq)
    _require(out, "out", (torch.float32,), b * hq * d)
    _require(workspace, "workspace", (torch.uint8,))
    ks = _scales_ptr(params, k_scales, k_codes)
    vp = ctypes.c_void_p
    args = (ctypes.byref(params.c), ctypes.byref(layout.c), vp(q.data_ptr()), ctypes.c_int(_dtype_code(q)),
            ctypes.c_int32(b), ctypes.c_int32(hq), vp(k_codes.data_ptr()), vp(v_codes.data_ptr()),
            vp(ks), vp(_sq_ptr(params, v_sq, k_codes)), _band_ref(band, params, b), vp(seq_lens.data_ptr()),
            ctypes.c_int32(max_seq_len),
            ctypes.c_int32(window),
            vp(sinks.data_ptr() if sinks is not None else None), ctypes.c_float(softmax_scale),
            vp(out.data_ptr()), vp(workspace.data_ptr()), ctypes.c_size_t(workspace.numel()),
            vp(_stream_ptr(stream)))
    return PreparedCall(nat.lib().nova_kv_decode_attn, args,
                        (params, layout, q, k_codes, v_codes, seq_lens, sinks, out, workspace, k_scales, band,
                         v_sq))


def prepare_append_decode(params: NovaKVParams, layout: CacheLayout, k_new: torch.Tensor, v_new: torch.Tensor,
                          q: torch.Tensor, k_codes: torch.Tensor, v_codes: torch.Tensor,
                          seq_lens: torch.Tensor, max_seq_len: int, out: torch.Tensor, workspace: torch.Tensor,
                          window: int = 0, sinks: Optional[torch.Tensor] = None, softmax_scale: float = 0.0,
                          stream: Optional[torch.cuda.Stream] = None,
                          k_scales: Optional[torch.Tensor] = None, band: Optional[Band] = None,
                          v_sq: Optional[torch.Tensor] = None) -> PreparedCall:
    """nova_kv_append_decode_attn with the arguments of append_decode_attn(),
    marshalled once (out and a zero-filled workspace are required here)."""
    args = _append_decode_args(params, layout, k_new, v_new, q, k_codes, v_codes, seq_lens, max_seq_len, out,
                               workspace, window, sinks, softmax_scale, stream, k_scales, band, v_sq)
    return PreparedCall(nat.lib().nova_kv_append_decode_attn, args,
                        (params, layout, k_new, v_new, q, k_codes, v_codes, seq_lens, sinks, out, workspace,
                         k_scales, band, v_sq))
