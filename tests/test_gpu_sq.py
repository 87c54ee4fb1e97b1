"""GPU parity of the scalar value arm (values as per-token affine INT2 in the
rotation t_v, with bf16 scale and offset).

* encode: key codes bit-exact except near-ties; value codes, scales and
  offsets equal to the oracle's except at rounding boundaries (an unrounded
  code within 1e-9 of a half-integer, a scale or offset within 1e-12
  relative of a bf16 rounding boundary);
* decode (the head_dim-128 table kernel, the split-K kernels at head_dim 64):
  max-abs error within 2e-3 of each output row's L2 norm, with windows,
  sinks, the key-scale format, fp8 key codebooks and the band.
"""

import numpy as np
import pytest
import torch

import synth
from helpers import assert_outputs_close, compare_codes, pool_offsets, read_rows, write_rows
from oracle import attention as oatt
from oracle import codec as ocodec
from oracle_cache import calibrated_params

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


@pytest.fixture(scope="module")
def nk():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_04074_amd as nk
    nk._native.lib()          # fail loudly if the HIP library is missing
    return nk


def dev(x, dtype):
    return torch.as_tensor(np.ascontiguousarray(x)).to(dtype).cuda()


def dev_bits(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


def sq_params(nk, wl, key_scale=False):
    params = calibrated_params(wl, 0, key_scale=key_scale)
    return params, nk.NovaKVParams.from_arrays(dict(params, cb_v=None), key_scale=key_scale, sq_values=True)


def near_bits(bits, x):
    """bf16 bits of x, or of x nudged by 1e-12 relative either way."""
    return ((bits == ocodec.bf16_bits(x)) | (bits == ocodec.bf16_bits(x * (1 - 1e-12)))
            | (bits == ocodec.bf16_bits(x * (1 + 1e-12))))


def compare_sq(gpu_packed, gpu_scale, gpu_zero, v, t_v, what):
    """Value codes, scales and offsets of the GPU against the oracle's, up to rounding boundaries."""
    packed, sb, zb = ocodec.sq_encode_values(v, t_v)
    s = ocodec.value_coefficients(v, t_v)
    mn, mx = s.min(axis=1), s.max(axis=1)
    ok_s = near_bits(gpu_scale, (mx - mn) / 3.0)
    ok_z = near_bits(gpu_zero, mn)
    assert ok_s.all() and ok_z.all(), f"{what}: scale/offset mismatches away from rounding boundaries"
    same = (gpu_scale == sb) & (gpu_zero == zb)
    q_gpu = ocodec.sq_unpack(gpu_packed)[same]
    q_ref = ocodec.sq_unpack(packed)[same]
    scale = ocodec.bf16_value(sb)[same][:, None]
    zero = ocodec.bf16_value(zb)[same][:, None]
    with np.errstate(divide="ignore", invalid="ignore"):
        u = np.where(scale > 0, (s[same] - zero) / scale, 0.0)
    near = np.abs(u - np.floor(u) - 0.5) < 1e-9
    bad = (q_gpu != q_ref) & ~near
    print(f"[parity] {what} tokens={len(sb)} scale/offset boundary cases={int((~same).sum())} "
          f"code mismatches={int((q_gpu != q_ref).sum())}", flush=True)
    assert not bad.any(), f"{what}: {int(bad.sum())} value code mismatches away from rounding boundaries"


@pytest.mark.parametrize("shape,n_new,paged,dtype", [("qwen3_8b", 1100, False, "bf16"), ("qwen3_8b", 3, True, "bf16"),
                                                     ("gptoss_pair", 40, False, "f32"), ("gptoss_pair", 1, False, "f32")])
def test_encode(nk, shape, n_new, paged, dtype):
    wl = synth.get_workload(shape)
    params, P = sq_params(nk, wl)
    B, start, cap = 2, 37, 1280
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    kk = np.empty((B, n_new, H, D))
    vv = np.empty_like(kk)
    for b in range(B):
        for kv in range(H):
            kk[b, :, kv], vv[b, :, kv] = synth.cache_tokens(wl, 0, kv, b, n_new)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    if dtype == "f32":  # fp32 inputs off the bf16 grid
        rng = np.random.default_rng(8)
        kk = (kk + 1e-3 * rng.standard_normal(kk.shape)).astype(np.float32).astype(np.float64)
        vv = (vv + 1e-3 * rng.standard_normal(vv.shape)).astype(np.float32).astype(np.float64)
    if paged:
        bs, bps = 16, cap // 16
        table = np.random.default_rng(7).permutation(B * bps).astype(np.int32).reshape(B, bps)
        lay = nk.CacheLayout(bs, bps, dev(table, torch.int32))
    else:
        bs, bps, table = cap, 1, None
        lay = nk.CacheLayout.contiguous(cap)
    lk = dict(hkv=H, block_size=bs, blocks_per_seq=bps, table=table)
    pk = torch.zeros((B * bps, H, bs, L), dtype=torch.uint8, device="cuda")
    pv = torch.zeros_like(pk)
    psq = torch.zeros((B * bps, H, bs, 2), dtype=torch.int16, device="cuda")
    say(f"sq encode {shape} n_new={n_new} paged={paged} {dtype}")
    nk.encode(P, lay, dev(kk, tdt), dev(vv, tdt), dev([start] * B, torch.int32), pk, pv, v_sq=psq)
    torch.cuda.synchronize()
    hk, hv = pk.cpu().numpy().reshape(-1), pv.cpu().numpy().reshape(-1)
    hs = psq.cpu().numpy().view(np.uint16).reshape(-1, 2)
    for b in range(B):
        for kv in range(H):
            hp = oatt.head_params(params, kv)
            ck, gk, _, _ = ocodec.encode_tokens(kk[b, :, kv], vv[b, :, kv], hp)
            compare_codes(read_rows(hk, b, kv, start, n_new, groups=L, **lk), ck, gk, f"sq b{b} kv{kv} K")
            rows = pool_offsets(b, kv, np.arange(start, start + n_new), groups=1, **lk)
            compare_sq(read_rows(hv, b, kv, start, n_new, groups=L, **lk), hs[rows, 0], hs[rows, 1],
                       vv[b, :, kv], hp["t_v"], f"sq b{b} kv{kv} V")
    assert not read_rows(hv, 0, 0, 0, start, groups=L, **lk).any()


def _random_sq_cache(wl, B, cap, H, L, seed=0):
    rng = np.random.default_rng(seed)
    ck = synth.random_codes(wl, 0, "k", (B, H, cap, L))
    cv = rng.integers(0, 256, (B, H, cap, L), dtype=np.uint8)           # four random 2-bit codes per byte
    sb = synth.random_key_scales(wl, 0, (B, H, cap), sigma=0.3)          # positive bf16 scales
    zb = ocodec.bf16_bits(-1.5 * ocodec.bf16_value(sb) + 0.2 * rng.standard_normal((B, H, cap)))
    return ck, cv, sb, zb


def _sq_decode_case(nk, wl, params, P, lens, cap, *, window=0, sinks=None, key_scale=False, band=None, what=""):
    B = len(lens)
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    ck, cv, sb, zb = _random_sq_cache(wl, B, cap, H, L)
    vsq = np.stack([sb, zb], axis=-1)
    ks = synth.random_key_scales(wl, 0, (B, H, cap)) if key_scale else None
    q = synth.decode_queries(wl, 0, batch=B)
    kw = {}
    exact = None
    if band is not None:
        n_sink, n_rec = band
        bk = np.full((B, H, n_sink + n_rec, D), 0x7FC0, dtype=np.uint16)
        bv = bk.copy()
        exact = {}
        for b in range(B):
            S = int(lens[b])
            for kv in range(H):
                kx, vx = synth.cache_tokens(wl, 0, kv, b, max(S, 1))
                exact[b, kv] = (ocodec.band_values(kx), ocodec.band_values(vx))
                for p in np.flatnonzero(oatt.band_mask(S, n_sink, n_rec)):
                    sl = p if p < n_sink else n_sink + p % n_rec
                    bk[b, kv, sl] = ocodec.bf16_bits(kx[p])
                    bv[b, kv, sl] = ocodec.bf16_bits(vx[p])
        kw["band"] = nk.Band(n_sink, n_rec, dev_bits(bk), dev_bits(bv))
    say(f"sq decode {what}")
    out = nk.decode_attn(P, nk.CacheLayout.contiguous(cap), dev(q, torch.bfloat16), dev(ck, torch.uint8),
                         dev(cv, torch.uint8), dev(np.asarray(lens, dtype=np.int32), torch.int32), cap,
                         window=window, sinks=dev(sinks, torch.float32) if sinks is not None else None,
                         k_scales=dev_bits(ks) if key_scale else None, v_sq=dev_bits(vsq), **kw).cpu().numpy()
    assert np.isfinite(out).all()
    scale = 1 / np.sqrt(D)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        S = int(lens[b])
        for kv in range(H):
            heads = slice(kv * G, (kv + 1) * G)
            bnd = None
            if band is not None:
                kb, vb = exact[b, kv]
                bnd = (band[0], band[1], kb[:S], vb[:S])
            ref[b, heads] = oatt.decode_rows(q[b, heads], ck[b, kv, :S], cv[b, kv, :S], oatt.head_params(params, kv),
                                             scale, window, None if sinks is None else sinks[heads],
                                             scales_k=ocodec.bf16_value(ks[b, kv, :S]) if key_scale else None,
                                             band=bnd, sq_v=(sb[b, kv, :S], zb[b, kv, :S]))
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D), what=f"sq {what}")


@pytest.mark.parametrize("window,use_sink", [(0, False), (300, True), (1, False)])
def test_qwen_shape_decode(nk, window, use_sink):
    wl = synth.get_workload("qwen3_8b")
    params, P = sq_params(nk, wl)
    sinks = np.random.default_rng(3).standard_normal(wl.num_q_heads).astype(np.float32) if use_sink else None
    _sq_decode_case(nk, wl, params, P, [0, 1, 255, 1023, 2000, 2304], 2304, window=window, sinks=sinks,
                    what=f"qwen window={window} sink={use_sink}")


def test_qwen_shape_decode_with_key_scale_and_band(nk):
    wl = synth.get_workload("qwen3_8b")
    params, P = sq_params(nk, wl, key_scale=True)
    _sq_decode_case(nk, wl, params, P, [2304, 700, 40], 2304, key_scale=True, band=(64, 256),
                    what="qwen key-scale + band")


@pytest.mark.parametrize("window", [0, 128])
def test_gptoss_shape_decode(nk, window):
    wl = synth.get_workload("gptoss_pair")
    params, P = sq_params(nk, wl)
    _sq_decode_case(nk, wl, params, P, [2048, 1500, 129, 1], 2048, window=window, sinks=synth.sink_logits(wl, 0),
                    what=f"gptoss window={window}")


def test_qwen3_8b_full_size_sampled(nk):
    wl = synth.get_workload("qwen3_8b")
    params, P = sq_params(nk, wl)
    B, cap = wl.batch, wl.seq_len
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    ck, cv, sb, zb = _random_sq_cache(wl, B, cap, H, L, seed=5)
    q = synth.decode_queries(wl, 0, batch=B)
    say(f"sq qwen full decode B={B} S={cap}")
    out = nk.decode_attn(P, nk.CacheLayout.contiguous(cap), dev(q, torch.bfloat16), dev(ck, torch.uint8),
                         dev(cv, torch.uint8), dev(np.full(B, cap), torch.int32), cap,
                         v_sq=dev_bits(np.stack([sb, zb], axis=-1))).cpu().numpy()
    scale = 1 / np.sqrt(D)
    gots, refs = [], []
    for b, kv in [(0, 0), (3, 5), (7, 7)]:
        heads = slice(kv * G, (kv + 1) * G)
        refs.append(oatt.decode_rows(q[b, heads], ck[b, kv], cv[b, kv], oatt.head_params(params, kv), scale,
                                     sq_v=(sb[b, kv], zb[b, kv])))
        gots.append(out[b, heads])
    assert_outputs_close(np.concatenate(gots), np.concatenate(refs), what="sq qwen3_8b full")


def test_append_decode(nk):
    """The step call: the new token's key codes and value codes as the oracle's, the output as the oracle's."""
    wl = synth.get_workload("qwen3_8b")
    params, P = sq_params(nk, wl)
    B, cap = 4, 2048
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    lens = np.array([1, 65, 1500, 2048], dtype=np.int32)
    ck, cv, sb, zb = _random_sq_cache(wl, B, cap, H, L, seed=6)
    kn = np.empty((B, H, D))
    vn = np.empty_like(kn)
    for b in range(B):
        for kv in range(H):
            kn[b, kv], vn[b, kv] = (x[0] for x in synth.cache_tokens(wl, 0, kv, b, 1, start=int(lens[b]) - 1))
    q = synth.decode_queries(wl, 0, batch=B)
    pk, pv = dev(ck, torch.uint8), dev(cv, torch.uint8)
    psq = dev_bits(np.stack([sb, zb], axis=-1))
    say("sq append+decode")
    out = nk.append_decode_attn(P, nk.CacheLayout.contiguous(cap), dev(kn, torch.bfloat16), dev(vn, torch.bfloat16),
                                dev(q, torch.bfloat16), pk, pv, dev(lens, torch.int32), cap, v_sq=psq).cpu().numpy()
    hk, hv = pk.cpu().numpy(), pv.cpu().numpy()
    hs = psq.cpu().numpy().view(np.uint16)
    scale = 1 / np.sqrt(D)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        p = int(lens[b]) - 1
        for kv in range(H):
            hp = oatt.head_params(params, kv)
            okk, ogk, _, _ = ocodec.encode_tokens(kn[b, kv][None], vn[b, kv][None], hp)
            compare_codes(hk[b, kv, p:p + 1], okk, ogk, f"sq step b{b} kv{kv} K")
            compare_sq(hv[b, kv, p:p + 1], hs[b, kv, p:p + 1, 0], hs[b, kv, p:p + 1, 1], vn[b, kv][None], hp["t_v"],
                       f"sq step b{b} kv{kv} V")
            heads = slice(kv * G, (kv + 1) * G)
            ref[b, heads] = oatt.decode_rows(q[b, heads], hk[b, kv, :p + 1], hv[b, kv, :p + 1], hp, scale,
                                             sq_v=(hs[b, kv, :p + 1, 0], hs[b, kv, :p + 1, 1]))
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D), what="sq step")


def test_all_formats_together(nk):
    """Key scale, fp8 key codebooks, the band and the scalar value arm in one decode."""
    from oracle import fp8 as ofp8
    wl = synth.get_workload("qwen3_8b")
    params = calibrated_params(wl, 0, key_scale=True, fp8=True)
    b8 = dict(params, cb_k=ofp8.e4m3_bits(params["cb_k"].astype(np.float64)), cb_v=None)
    P = nk.NovaKVParams.from_arrays(b8, key_scale=True, sq_values=True)
    assert P.fp8_codebooks and P.key_scale and P.sq_values
    sinks = np.random.default_rng(4).standard_normal(wl.num_q_heads).astype(np.float32)
    _sq_decode_case(nk, wl, params, P, [2304, 1500, 300, 1], 2304, window=1000, sinks=sinks, key_scale=True,
                    band=(64, 256), what="qwen all formats")


@pytest.mark.parametrize("window", [0, 128])
def test_gptoss_deployed_format(nk, window):
    """The deployed format at the GPT-OSS shape (D = 64, eight query heads per
    KV head) on its table kernel: keys with a per-token scale, INT2 values,
    a 64 + 256 band and sinks; ragged lengths that leave splits empty."""
    wl = synth.get_workload("gptoss_pair")
    params, P = sq_params(nk, wl, key_scale=True)
    _sq_decode_case(nk, wl, params, P, [4096, 2500, 400, 257, 1], 4096, window=window,
                    sinks=synth.sink_logits(wl, 0), key_scale=True, band=(64, 256),
                    what=f"gptoss deployed format window={window}")
