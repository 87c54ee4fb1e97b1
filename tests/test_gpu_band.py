"""GPU parity of the sink-plus-recent band (first n_sink and last n_rec
positions held in BF16, the rest read from codes).

The HIP path (through the C ABI) against the fp64 CPU oracle:
* encode: the band rows written are the inputs' bf16 bit patterns, at the
  slots the layout names, and nothing else; the codes are those of the
  encode without a band;
* decode: max-abs error within 2e-3 of each output row's L2 norm, on every
  kernel family (head_dim 128 and 64 table kernels, the split-K kernels of
  8-token pages), with windows, sinks, the key-scale format, sequences
  shorter than the band, and the largest band; band slots that hold no
  attended position are filled with NaN, so reading one fails the test.
"""

import numpy as np
import pytest
import torch

import synth
from helpers import assert_outputs_close, pool_offsets, read_rows, write_rows
from oracle import attention as oatt
from oracle import codec as ocodec
from oracle_cache import calibrated_params

pytestmark = pytest.mark.gpu

NAN_BF16 = 0x7FC0


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


def slot(p, n_sink, n_rec):
    return p if p < n_sink else n_sink + p % n_rec


def band_positions(S, n_sink, n_rec):
    return np.flatnonzero(oatt.band_mask(S, n_sink, n_rec))


@pytest.fixture(scope="module")
def qwen(nk):
    wl = synth.get_workload("qwen3_8b")
    params = calibrated_params(wl, 0)
    return wl, params, nk.NovaKVParams.from_arrays(params)


@pytest.fixture(scope="module")
def gptoss(nk):
    wl = synth.get_workload("gptoss_pair")
    params = calibrated_params(wl, 0)
    return wl, params, nk.NovaKVParams.from_arrays(params)


# --------------------------------------------------------------------- encode

@pytest.mark.parametrize("n_new,start", [(1100, 37), (3, 600), (2, 10)])
def test_encode_writes_the_band(nk, qwen, n_new, start):
    """Band rows of the new tokens in the band after the append, bit for bit;
    every other slot untouched; codes as without a band."""
    wl, params, P = qwen
    B, cap, n_sink, n_rec = 2, 1280, 64, 256
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    kk = np.empty((B, n_new, H, D))
    vv = np.empty_like(kk)
    for b in range(B):
        for kv in range(H):
            kk[b, :, kv], vv[b, :, kv] = synth.cache_tokens(wl, 0, kv, b, n_new)
    lay = nk.CacheLayout.contiguous(cap)
    kd, vd, sp = dev(kk, torch.bfloat16), dev(vv, torch.bfloat16), dev([start] * B, torch.int32)
    pk0 = torch.zeros((B, H, cap, L), dtype=torch.uint8, device="cuda")
    pv0 = torch.zeros_like(pk0)
    nk.encode(P, lay, kd, vd, sp, pk0, pv0)
    pk, pv = torch.zeros_like(pk0), torch.zeros_like(pk0)
    shape = nk.band_shape(P, B, n_sink, n_rec)
    fill = np.full(shape, 0x1234, dtype=np.uint16)
    bk, bv = dev_bits(fill), dev_bits(fill)
    say(f"band encode n_new={n_new} start={start}")
    nk.encode(P, lay, kd, vd, sp, pk, pv, band=nk.Band(n_sink, n_rec, bk, bv))
    torch.cuda.synchronize()
    assert torch.equal(pk, pk0) and torch.equal(pv, pv0)
    hk = bk.cpu().numpy().view(np.uint16)
    hv = bv.cpu().numpy().view(np.uint16)
    ek, ev = fill.copy(), fill.copy()
    end = start + n_new
    for t in range(n_new):
        p = start + t
        if p < n_sink or p >= end - n_rec:
            s = slot(p, n_sink, n_rec)
            ek[:, :, s] = ocodec.bf16_bits(kk[:, t])
            ev[:, :, s] = ocodec.bf16_bits(vv[:, t])
    assert np.array_equal(hk, ek) and np.array_equal(hv, ev)


def test_encode_band_rounds_fp32_inputs(nk, gptoss):
    """fp32 inputs (D = 64): band rows are the inputs rounded to bf16, to nearest even."""
    wl, params, P = gptoss
    B, n_new, n_sink, n_rec = 2, 40, 4, 16
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    rng = np.random.default_rng(21)
    kk = rng.standard_normal((B, n_new, H, D)).astype(np.float32)
    vv = rng.standard_normal((B, n_new, H, D)).astype(np.float32)
    kk[0, 0, 0, :4] = [1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -2.0 ** -9, 3.0]   # ties and exact values
    lay = nk.CacheLayout.contiguous(256)
    pk = torch.zeros((B, H, 256, L), dtype=torch.uint8, device="cuda")
    pv = torch.zeros_like(pk)
    shape = nk.band_shape(P, B, n_sink, n_rec)
    bk = dev_bits(np.zeros(shape, dtype=np.uint16))
    bv = dev_bits(np.zeros(shape, dtype=np.uint16))
    say("band encode fp32 inputs, D=64")
    nk.encode(P, lay, dev(kk, torch.float32), dev(vv, torch.float32), dev([0, 100], torch.int32), pk, pv,
              band=nk.Band(n_sink, n_rec, bk, bv))
    torch.cuda.synchronize()
    hk = bk.cpu().numpy().view(np.uint16)
    hv = bv.cpu().numpy().view(np.uint16)
    for b, start in ((0, 0), (1, 100)):
        for t in range(n_new):
            p = start + t
            if p < n_sink or p >= start + n_new - n_rec:
                s = slot(p, n_sink, n_rec)
                assert np.array_equal(hk[b, :, s], ocodec.bf16_bits(kk[b, t].astype(np.float64)))
                assert np.array_equal(hv[b, :, s], ocodec.bf16_bits(vv[b, t].astype(np.float64)))


# --------------------------------------------------------------------- decode

def _band_case(nk, wl, params, P, lens, cap, n_sink, n_rec, *, window=0, sinks=None, paged_bs=None,
               key_scale=False, what=""):
    B = len(lens)
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    ck = synth.random_codes(wl, 0, "k", (B, H, cap, L))
    cv = synth.random_codes(wl, 0, "v", (B, H, cap, L))
    sk = synth.random_key_scales(wl, 0, (B, H, cap)) if key_scale else None
    if paged_bs:
        bps = cap // paged_bs
        table = np.random.default_rng(13).permutation(B * bps).astype(np.int32).reshape(B, bps)
        lk = dict(hkv=H, block_size=paged_bs, blocks_per_seq=bps, table=table)
        lay = nk.CacheLayout(paged_bs, bps, dev(table, torch.int32))
    else:
        lk = dict(hkv=H, block_size=cap, blocks_per_seq=1, table=None)
        lay = nk.CacheLayout.contiguous(cap)
    flat_k = np.zeros(B * lk["blocks_per_seq"] * H * lk["block_size"] * L, dtype=np.uint8)
    flat_v = np.zeros_like(flat_k)
    flat_s = np.zeros(flat_k.size // L, dtype=np.uint16)
    for b in range(B):
        for kv in range(H):
            write_rows(flat_k, ck[b, kv], b, kv, 0, **lk)
            write_rows(flat_v, cv[b, kv], b, kv, 0, **lk)
            if key_scale:
                flat_s[pool_offsets(b, kv, np.arange(cap), groups=1, **lk)] = sk[b, kv]
    # exact keys and values of every position (the band holds some of them);
    # slots with no attended band position hold NaN
    shape = (B, H, n_sink + n_rec, D)
    band_k = np.full(shape, NAN_BF16, dtype=np.uint16)
    band_v = np.full(shape, NAN_BF16, dtype=np.uint16)
    exact = {}
    for b in range(B):
        S = int(lens[b])
        for kv in range(H):
            kx, vx = synth.cache_tokens(wl, 0, kv, b, max(S, 1))
            exact[b, kv] = (ocodec.band_values(kx), ocodec.band_values(vx))
            lo = max(0, S - window) if window else 0
            for p in band_positions(S, n_sink, n_rec):
                if p >= lo:
                    band_k[b, kv, slot(p, n_sink, n_rec)] = ocodec.bf16_bits(kx[p])
                    band_v[b, kv, slot(p, n_sink, n_rec)] = ocodec.bf16_bits(vx[p])
    q = synth.decode_queries(wl, 0, batch=B)
    say(f"band decode {what}")
    out = nk.decode_attn(P, lay, dev(q, torch.bfloat16), dev(flat_k, torch.uint8), dev(flat_v, torch.uint8),
                         dev(np.asarray(lens, dtype=np.int32), torch.int32), cap, window=window,
                         sinks=dev(sinks, torch.float32) if sinks is not None else None,
                         k_scales=dev_bits(flat_s) if key_scale else None,
                         band=nk.Band(n_sink, n_rec, dev_bits(band_k), dev_bits(band_v))).cpu().numpy()
    assert np.isfinite(out).all()
    scale = 1 / np.sqrt(D)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        S = int(lens[b])
        for kv in range(H):
            kb, vb = exact[b, kv]
            rk = read_rows(flat_k, b, kv, 0, S, groups=L, **lk)
            rv = read_rows(flat_v, b, kv, 0, S, groups=L, **lk)
            rho = ocodec.bf16_value(sk[b, kv, :S]) if key_scale else None
            heads = slice(kv * G, (kv + 1) * G)
            ref[b, heads] = oatt.decode_rows(q[b, heads], rk, rv, oatt.head_params(params, kv), scale, window,
                                             None if sinks is None else sinks[heads], scales_k=rho,
                                             band=(n_sink, n_rec, kb[:S], vb[:S]))
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D), what=f"band {what}")
    return out


@pytest.mark.parametrize("paged,window,use_sink", [(False, 0, False), (False, 300, True), (True, 0, True),
                                                   (False, 1, False), (False, 100, False)])
def test_qwen_shape_decode(nk, qwen, paged, window, use_sink):
    """head_dim 128 table kernel: sequences shorter than the sink, inside the
    band, and long ones; windows that cut the band or fall inside it."""
    wl, params, P = qwen
    sinks = np.random.default_rng(3).standard_normal(wl.num_q_heads).astype(np.float32) if use_sink else None
    _band_case(nk, wl, params, P, [0, 1, 40, 255, 1500, 2304], 2304, 64, 256, window=window, sinks=sinks,
               paged_bs=16 if paged else None, what=f"qwen paged={paged} window={window} sink={use_sink}")


def test_qwen_shape_largest_band_and_sink_only(nk, qwen):
    """The largest band (1024 positions), and a band of sink positions only."""
    wl, params, P = qwen
    _band_case(nk, wl, params, P, [2304, 1100, 1023], 2304, 24, 1000, what="qwen band 24+1000")
    _band_case(nk, wl, params, P, [2304, 100, 7], 2304, 64, 0, what="qwen sink-only band 64+0")
    _band_case(nk, wl, params, P, [2304, 100, 7], 2304, 0, 128, what="qwen recent-only band 0+128")


def test_qwen_shape_key_scale_with_band(nk):
    wl = synth.get_workload("qwen3_8b")
    params = calibrated_params(wl, 0, key_scale=True)
    P = nk.NovaKVParams.from_arrays(params, key_scale=True)
    _band_case(nk, wl, params, P, [2304, 700, 200], 2304, 64, 256, key_scale=True, what="qwen key-scale")


@pytest.mark.parametrize("window", [0, 128])
def test_gptoss_shape_decode(nk, gptoss, window):
    """head_dim 64 table kernel, 8 query heads per KV head, sinks, a window inside the band."""
    wl, params, P = gptoss
    _band_case(nk, wl, params, P, [2048, 1500, 300, 1], 2048, 64, 256, window=window,
               sinks=synth.sink_logits(wl, 0), what=f"gptoss window={window}")


@pytest.mark.parametrize("window,use_sink", [(0, False), (200, True)])
def test_generic_path_block8_decode(nk, qwen, window, use_sink):
    """Pages of 8 tokens take the split-K kernels."""
    wl, params, P = qwen
    sinks = np.random.default_rng(31).standard_normal(wl.num_q_heads).astype(np.float32) if use_sink else None
    _band_case(nk, wl, params, P, [0, 9, 300, 1000], 1000, 64, 256, window=window, sinks=sinks, paged_bs=8,
               what=f"block8 window={window} sink={use_sink}")


def test_qwen3_8b_full_size_sampled(nk, qwen):
    """Qwen3-8B decode shape at full size (8 sequences x 16384 tokens) with the
    paper's band (64 + 256), sampled units against the oracle."""
    wl, params, P = qwen
    B, cap, n_sink, n_rec = wl.batch, wl.seq_len, 64, 256
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    ck = synth.random_codes(wl, 0, "k", (B, H, cap, L))
    cv = synth.random_codes(wl, 0, "v", (B, H, cap, L))
    units = [(0, 0), (3, 5), (7, 7)]
    band_k = np.full((B, H, n_sink + n_rec, D), NAN_BF16, dtype=np.uint16)
    band_v = band_k.copy()
    rng = np.random.default_rng(9)
    band_pos = band_positions(cap, n_sink, n_rec)
    slots = [slot(p, n_sink, n_rec) for p in band_pos]
    exact = {}
    for b in range(B):
        for kv in range(H):
            kx = ocodec.band_values(rng.standard_normal((n_sink + n_rec, D)))
            vx = ocodec.band_values(rng.standard_normal((n_sink + n_rec, D)))
            band_k[b, kv, slots] = ocodec.bf16_bits(kx)
            band_v[b, kv, slots] = ocodec.bf16_bits(vx)
            exact[b, kv] = (kx, vx)
    q = synth.decode_queries(wl, 0, batch=B)
    lens = np.full(B, cap, dtype=np.int32)
    say(f"band qwen full decode B={B} S={cap}")
    out = nk.decode_attn(P, nk.CacheLayout.contiguous(cap), dev(q, torch.bfloat16), dev(ck, torch.uint8),
                         dev(cv, torch.uint8), dev(lens, torch.int32), cap,
                         band=nk.Band(n_sink, n_rec, dev_bits(band_k), dev_bits(band_v))).cpu().numpy()
    assert np.isfinite(out).all()
    scale = 1 / np.sqrt(D)
    gots, refs = [], []
    for b, kv in units:
        kx, vx = exact[b, kv]
        kf = np.zeros((cap, D))
        vf = np.zeros((cap, D))
        kf[band_pos], vf[band_pos] = kx, vx
        heads = slice(kv * G, (kv + 1) * G)
        refs.append(oatt.decode_rows(q[b, heads], ck[b, kv], cv[b, kv], oatt.head_params(params, kv), scale,
                                     band=(n_sink, n_rec, kf, vf)))
        gots.append(out[b, heads])
    assert_outputs_close(np.concatenate(gots), np.concatenate(refs), what="band qwen3_8b full")


@pytest.mark.parametrize("shape", ["qwen3_8b", "gptoss_pair"])
def test_append_decode(nk, qwen, gptoss, shape):
    """The step call with a band: the new token's band row and codes as the
    encoder's, the output as the oracle's over the cache with it."""
    wl, params, P = qwen if shape == "qwen3_8b" else gptoss
    B, cap, n_sink, n_rec = 4, 2048, 64, 256
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    lens = np.array([1, 65, 400, 2048], dtype=np.int32)
    ck = synth.random_codes(wl, 0, "k", (B, H, cap, L))
    cv = synth.random_codes(wl, 0, "v", (B, H, cap, L))
    shape_b = (B, H, n_sink + n_rec, D)
    band_k = np.full(shape_b, NAN_BF16, dtype=np.uint16)
    band_v = band_k.copy()
    exact = {}
    for b in range(B):
        S = int(lens[b])
        for kv in range(H):
            kx, vx = synth.cache_tokens(wl, 0, kv, b, S)
            exact[b, kv] = (ocodec.band_values(kx), ocodec.band_values(vx))
            for p in band_positions(S - 1, n_sink, n_rec):   # the band before the step's token
                band_k[b, kv, slot(p, n_sink, n_rec)] = ocodec.bf16_bits(kx[p])
                band_v[b, kv, slot(p, n_sink, n_rec)] = ocodec.bf16_bits(vx[p])
    kn = np.stack([[exact[b, kv][0][int(lens[b]) - 1] for kv in range(H)] for b in range(B)])
    vn = np.stack([[exact[b, kv][1][int(lens[b]) - 1] for kv in range(H)] for b in range(B)])
    q = synth.decode_queries(wl, 0, batch=B)
    sinks = synth.sink_logits(wl, 0)
    pk, pv = dev(ck, torch.uint8), dev(cv, torch.uint8)
    bk, bv = dev_bits(band_k), dev_bits(band_v)
    say(f"band append+decode {shape}")
    out = nk.append_decode_attn(P, nk.CacheLayout.contiguous(cap), dev(kn, torch.bfloat16), dev(vn, torch.bfloat16),
                                dev(q, torch.bfloat16), pk, pv, dev(lens, torch.int32), cap,
                                sinks=dev(sinks, torch.float32) if sinks is not None else None,
                                band=nk.Band(n_sink, n_rec, bk, bv)).cpu().numpy()
    hk = pk.cpu().numpy()
    hbk = bk.cpu().numpy().view(np.uint16)
    scale = 1 / np.sqrt(D)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        S = int(lens[b])
        p = S - 1
        for kv in range(H):
            kb, vb = exact[b, kv]
            assert np.array_equal(hbk[b, kv, slot(p, n_sink, n_rec)], ocodec.bf16_bits(kb[p]))
            okk, _, ovv, _ = ocodec.encode_tokens(kb[p][None], vb[p][None], oatt.head_params(params, kv))
            rk = hk[b, kv, :S].copy()
            rv = cv[b, kv, :S].copy()
            rv[p] = ovv[0]
            heads = slice(kv * G, (kv + 1) * G)
            ref[b, heads] = oatt.decode_rows(q[b, heads], rk, rv, oatt.head_params(params, kv), scale, 0,
                                             None if sinks is None else sinks[heads],
                                             band=(n_sink, n_rec, kb, vb))
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D), what=f"band step {shape}")


def test_many_splits_share_the_band(nk, qwen):
    """One sequence of 16384 tokens: 32 splits, each attending about ten band
    rows, with the band cut by a window and a sink."""
    wl, params, P = qwen
    sinks = np.random.default_rng(12).standard_normal(wl.num_q_heads).astype(np.float32)
    _band_case(nk, wl, params, P, [16384], 16384, 64, 256, what="qwen B=1 S=16384 (32 splits)")
    _band_case(nk, wl, params, P, [16384], 16384, 64, 256, window=16300, sinks=sinks,
               what="qwen B=1 S=16384 window 16300")


def test_split_groups_share_the_band(nk, qwen):
    """One KV head of one sequence at 65536 tokens: 128 splits, merged in
    groups before the final combine, each group carrying its splits' band
    shares (a window cuts the band)."""
    wl0, params0, _ = qwen
    wl = wl0.scaled(num_kv_heads=1, num_q_heads=wl0.gqa)
    params = {k: v[:1] for k, v in params0.items()}
    P = nk.NovaKVParams.from_arrays(params)
    sinks = np.random.default_rng(14).standard_normal(wl.num_q_heads).astype(np.float32)
    _band_case(nk, wl, params, P, [65536], 65536, 64, 256, sinks=sinks, what="one KV head S=65536 (128 splits)")
    _band_case(nk, wl, params, P, [65536], 65536, 64, 256, window=65000,
               what="one KV head S=65536 window 65000")
