"""C-ABI checks that need no GPU: exports, status strings, host-side argument validation.

Every call here is rejected by the host-side checks before any HIP call or
launch, so nothing touches a device.
"""

import ctypes
import os
import re

import pytest

from paper_2608_04074_amd import _native as nat

NOALLOC_BYTES = 32 << 20   # the allocation-free step's fixed scratch array

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "nova_kv.h")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(nova_kv_\w+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    lib = nat.lib()
    declared = _declared_functions()
    assert set(declared) == set(nat.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings():
    lib = nat.lib()
    for s in range(5):
        assert lib.nova_kv_status_string(s)
    assert lib.nova_kv_status_string(99) == b"unknown status"


def _band(b):
    """(n_sink, n_rec, k, v) -> a pointer to a nova_kv_band, or NULL."""
    return None if b is None else ctypes.byref(nat.Band(*b))


def _params(**kw):
    base = dict(num_kv_heads=8, head_dim=128, group_dim=4, codebook_size=256, flags=0,
                kbar=0x1000, t_k=0x2000, t_k_inv_t=0x3000, t_v=0x4000, cb_k=0x5000, cb_v=0x6000)
    base.update(kw)
    return nat.Params(**base)


def _layout(**kw):
    base = dict(block_size=4096, blocks_per_seq=1, block_table=None)
    base.update(kw)
    return nat.Layout(**base)


def _decode(p, lay, **kw):
    a = dict(q=0x7000, q_dtype=nat.NOVA_KV_BF16, batch=2, hq=32, k=0x8000, v=0x9000, seq=0xA000,
             max_seq=4096, window=0, sinks=None, scale=0.0, out=0xB000, ws=None, ws_bytes=0, ks=None,
             vsq=None, band=None)
    a.update(kw)
    return nat.lib().nova_kv_decode_attn(
        ctypes.byref(p) if p is not None else None, ctypes.byref(lay) if lay is not None else None,
        a["q"], a["q_dtype"], a["batch"], a["hq"], a["k"], a["v"], a["ks"], a["vsq"], _band(a["band"]), a["seq"],
        a["max_seq"],
        a["window"], a["sinks"], a["scale"], a["out"], a["ws"], a["ws_bytes"], None)


def _encode(p, lay, **kw):
    a = dict(k=0x7000, v=0x7800, dtype=nat.NOVA_KV_BF16, batch=2, n_new=16, start=0xA000,
             kc=0x8000, vc=0x9000, ks=None, vsq=None, band=None)
    a.update(kw)
    return nat.lib().nova_kv_encode(ctypes.byref(p) if p is not None else None,
                                    ctypes.byref(lay) if lay is not None else None,
                                    a["k"], a["v"], a["dtype"], a["batch"], a["n_new"], a["start"],
                                    a["kc"], a["vc"], a["ks"], a["vsq"], _band(a["band"]), None)


@pytest.mark.parametrize("kw,status", [
    (dict(group_dim=8), nat.NOVA_KV_ERR_UNSUPPORTED),
    (dict(codebook_size=16), nat.NOVA_KV_ERR_UNSUPPORTED),
    (dict(head_dim=96), nat.NOVA_KV_ERR_UNSUPPORTED),
    (dict(head_dim=130), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(flags=16), nat.NOVA_KV_ERR_UNSUPPORTED),
    (dict(flags=31), nat.NOVA_KV_ERR_UNSUPPORTED),
    (dict(num_kv_heads=0), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(cb_k=None), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(cb_v=0x6001), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(t_k_inv_t=None), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(t_v=0x4004), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(kbar=0x1008), nat.NOVA_KV_ERR_INVALID_ARG),
])
def test_decode_rejects_bad_params(kw, status):
    assert _decode(_params(**kw), _layout()) == status
    assert nat.lib().nova_kv_last_error()


@pytest.mark.parametrize("kw,status", [
    (dict(hq=12), nat.NOVA_KV_ERR_INVALID_ARG),          # not a multiple of Hkv
    (dict(hq=128), nat.NOVA_KV_ERR_UNSUPPORTED),         # 16 query heads per KV head
    (dict(batch=-1), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(max_seq=0), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(max_seq=5000), nat.NOVA_KV_ERR_INVALID_ARG),   # above capacity 4096
    (dict(window=-3), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(q_dtype=7), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(scale=-1.0), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(q=None), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(out=None), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(k=0x8001), nat.NOVA_KV_ERR_INVALID_ARG),       # misaligned pool
    (dict(ws=None), nat.NOVA_KV_ERR_WORKSPACE),
    (dict(ws=0x10000, ws_bytes=16), nat.NOVA_KV_ERR_WORKSPACE),
    (dict(ws=0x10010, ws_bytes=1 << 30), nat.NOVA_KV_ERR_WORKSPACE),   # misaligned workspace
])
def test_decode_rejects_bad_arguments(kw, status):
    assert _decode(_params(), _layout(), **kw) == status


def test_decode_rejects_null_structs_and_bad_layout():
    assert _decode(None, _layout()) == nat.NOVA_KV_ERR_INVALID_ARG
    assert _decode(_params(), None) == nat.NOVA_KV_ERR_INVALID_ARG
    assert _decode(_params(), _layout(block_size=0)) == nat.NOVA_KV_ERR_INVALID_ARG


def test_decode_batch_zero_is_a_noop():
    assert _decode(_params(), _layout(), batch=0, q=None, out=None) == nat.NOVA_KV_OK


def test_workspace_query():
    lib = nat.lib()
    p = _params()
    n = lib.nova_kv_decode_workspace_bytes(ctypes.byref(p), 8, 32, 16384)
    assert n > 8 * 32 * 128 * 4 and n % 256 == 0
    assert lib.nova_kv_decode_workspace_bytes(ctypes.byref(p), 0, 32, 16384) == 0
    assert lib.nova_kv_decode_workspace_bytes(None, 8, 32, 16384) == 0
    # monotone in the context length
    assert lib.nova_kv_decode_workspace_bytes(ctypes.byref(p), 8, 32, 32768) >= n


@pytest.mark.parametrize("kw,status", [
    (dict(batch=-1), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(n_new=-1), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(n_new=5000), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(dtype=5), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(k=None), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(start=None), nat.NOVA_KV_ERR_INVALID_ARG),
    (dict(kc=None), nat.NOVA_KV_ERR_INVALID_ARG),
])
def test_encode_rejects_bad_arguments(kw, status):
    assert _encode(_params(), _layout(), **kw) == status


def test_encode_needs_forward_transforms_and_noops():
    assert _encode(_params(t_k=None), _layout()) == nat.NOVA_KV_ERR_INVALID_ARG
    assert _encode(_params(), _layout(), n_new=0, k=None) == nat.NOVA_KV_OK
    assert _encode(_params(), _layout(), batch=0, k=None) == nat.NOVA_KV_OK


def _append(p, lay, **kw):
    a = dict(kn=0x7000, vn=0x7800, new_dtype=nat.NOVA_KV_BF16, q=0x7400, q_dtype=nat.NOVA_KV_BF16,
             batch=2, hq=32, k=0x8000, v=0x9000, ks=None, vsq=None, band=None, seq=0xA000, max_seq=4096,
             window=0,
             sinks=None, scale=0.0, out=0xB000, ws=None, ws_bytes=0)
    a.update(kw)
    return nat.lib().nova_kv_append_decode_attn(
        ctypes.byref(p), ctypes.byref(lay), a["kn"], a["vn"], a["new_dtype"], a["q"], a["q_dtype"],
        a["batch"], a["hq"], a["k"], a["v"], a["ks"], a["vsq"], _band(a["band"]), a["seq"], a["max_seq"],
        a["window"],
        a["sinks"],
        a["scale"], a["out"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("call", [_decode, _encode, _append])
def test_key_scale_format_needs_an_aligned_scale_pool(call):
    p = _params(flags=nat.NOVA_KV_KEY_SCALE)
    assert call(p, _layout()) == nat.NOVA_KV_ERR_INVALID_ARG
    assert b"k_scales" in nat.lib().nova_kv_last_error()
    assert call(p, _layout(), ks=0xC001) == nat.NOVA_KV_ERR_INVALID_ARG
    # with a scale pool the checks go on to the next argument (no workspace;
    # for the encode a NULL input, so that nothing is launched)
    if call is _encode:
        assert call(p, _layout(), ks=0xC000, k=None) == nat.NOVA_KV_ERR_INVALID_ARG
        assert b"k_scales" not in nat.lib().nova_kv_last_error()
    else:
        assert call(p, _layout(), ks=0xC000) == nat.NOVA_KV_ERR_WORKSPACE
        # the plain format ignores the pointer
        assert call(_params(), _layout(), ks=0xC001) == nat.NOVA_KV_ERR_WORKSPACE
    # batch 0 stays a no-op
    assert call(p, _layout(), batch=0, q=None, out=None) == nat.NOVA_KV_OK


def test_append_rejects_bad_new_dtype():
    assert _append(_params(), _layout(), new_dtype=9) == nat.NOVA_KV_ERR_INVALID_ARG


@pytest.mark.parametrize("call", [_decode, _encode, _append])
@pytest.mark.parametrize("band", [(0, 0, 0xC000, 0xD000), (-1, 8, 0xC000, 0xD000), (64, 961, 0xC000, 0xD000),
                                  (64, 256, None, 0xD000), (64, 256, 0xC000, None), (64, 256, 0xC008, 0xD000)])
def test_bad_band_is_rejected(call, band):
    assert call(_params(), _layout(), band=band) == nat.NOVA_KV_ERR_INVALID_ARG
    assert b"band" in nat.lib().nova_kv_last_error()


@pytest.mark.parametrize("call", [_decode, _append])
def test_good_band_passes_the_checks(call):
    # the checks go on to the next argument: no workspace
    assert call(_params(), _layout(), band=(64, 256, 0xC000, 0xD000)) == nat.NOVA_KV_ERR_WORKSPACE
    assert call(_params(), _layout(), band=(0, 1024, 0xC000, 0xD000)) == nat.NOVA_KV_ERR_WORKSPACE
    # batch 0 stays a no-op whatever the band
    assert call(_params(), _layout(), band=(0, 0, None, None), batch=0, q=None, out=None) == nat.NOVA_KV_OK


@pytest.mark.parametrize("call", [_decode, _encode, _append])
def test_scalar_value_arm_needs_its_pool(call):
    p = _params(flags=nat.NOVA_KV_SQ_VALUES, cb_v=None)   # cb_v unused in this format
    assert call(p, _layout()) == nat.NOVA_KV_ERR_INVALID_ARG
    assert b"v_sq" in nat.lib().nova_kv_last_error()
    assert call(p, _layout(), vsq=0xC002) == nat.NOVA_KV_ERR_INVALID_ARG    # not 4-byte aligned
    if call is _encode:
        assert call(p, _layout(), vsq=0xC000, k=None) == nat.NOVA_KV_ERR_INVALID_ARG
        assert b"v_sq" not in nat.lib().nova_kv_last_error()
    else:
        assert call(p, _layout(), vsq=0xC000) == nat.NOVA_KV_ERR_WORKSPACE
    # the plain format still needs cb_v
    assert call(_params(cb_v=None), _layout()) == nat.NOVA_KV_ERR_INVALID_ARG


def _append_noalloc(p, lay, **kw):
    a = dict(kn=0x7000, vn=0x7800, new_dtype=nat.NOVA_KV_BF16, q=0x7400, q_dtype=nat.NOVA_KV_BF16,
             batch=2, hq=32, k=0x8000, v=0x9000, ks=None, vsq=None, band=None, seq=0xA000, max_seq=4096,
             window=0, sinks=None, scale=0.0, out=0xB000)
    a.update(kw)
    return nat.lib().nova_kv_append_decode_attn_noalloc(
        ctypes.byref(p), ctypes.byref(lay), a["kn"], a["vn"], a["new_dtype"], a["q"], a["q_dtype"],
        a["batch"], a["hq"], a["k"], a["v"], a["ks"], a["vsq"], _band(a["band"]), a["seq"], a["max_seq"],
        a["window"], a["sinks"], a["scale"], a["out"], None)


def test_noalloc_step_checks_before_any_hip_call():
    """The allocation-free step validates like the step with a workspace, and
    rejects a shape whose scratch exceeds its fixed array, all on the host."""
    lib = nat.lib()
    assert _append_noalloc(_params(), _layout(), new_dtype=9) == nat.NOVA_KV_ERR_INVALID_ARG
    assert _append_noalloc(_params(), _layout(), q=None) == nat.NOVA_KV_ERR_INVALID_ARG
    assert _append_noalloc(_params(), _layout(), kn=None) == nat.NOVA_KV_ERR_INVALID_ARG
    assert _append_noalloc(_params(), _layout(), batch=0, q=None, out=None) == nat.NOVA_KV_OK
    # 64 sequences of 32768 tokens need more scratch than the array holds
    big = _layout(block_size=32768)
    need = lib.nova_kv_decode_workspace_bytes(ctypes.byref(_params()), 64, 32, 32768)
    assert need > NOALLOC_BYTES
    assert _append_noalloc(_params(), big, batch=64, max_seq=32768) == nat.NOVA_KV_ERR_WORKSPACE
    msg = lib.nova_kv_last_error()
    assert b"allocation-free" in msg and str(NOALLOC_BYTES).encode() in msg
