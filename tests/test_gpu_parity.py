"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle.

Inputs are seeded synthetic workloads from ``synth``; transforms and codebooks
come from the oracle's calibration.  Codes must match bit-exactly except where
the oracle's top-2 distance gap is a near-tie (< 1e-6); decode outputs must
be within 2e-3 of the oracle's, max-abs relative to each row's L2 norm.
At full sizes the oracle checks sampled (sequence, KV head) units.
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


def qdtype(wl):
    return torch.float32 if wl.dtype == "f32" else torch.bfloat16


def upload_params(nk, params):
    return nk.NovaKVParams.from_arrays(params)


def lay_kwargs(wl_hkv, block_size, blocks_per_seq, table=None):
    return dict(hkv=wl_hkv, block_size=block_size, blocks_per_seq=blocks_per_seq, table=table)


def oracle_rows(q, pool_k, pool_v, params, b, kv, n, scale, lay, window=0, sinks=None, gqa=1):
    L = params["cb_k"].shape[1]
    ck = read_rows(pool_k, b, kv, 0, n, groups=L, **lay)
    cv = read_rows(pool_v, b, kv, 0, n, groups=L, **lay)
    hp = oatt.head_params(params, kv)
    heads = slice(kv * gqa, (kv + 1) * gqa)
    return oatt.decode_rows(q[b, heads], ck, cv, hp, scale, window,
                            None if sinks is None else sinks[heads])


# ----------------------------------------------------------------- config 1

def test_single_head_encode_and_decode(nk):
    """Single head, batch 1, D=128, S=2048, fp32: codes bit-exact, output within tolerance."""
    wl = synth.get_workload("single_head")
    params = calibrated_params(wl, 0)
    hp = oatt.head_params(params, 0)
    S, L = wl.seq_len, wl.groups
    kc, vc = synth.cache_tokens(wl, 0, 0, 0, S)
    P = upload_params(nk, params)
    lay = nk.CacheLayout.contiguous(S)
    pk = torch.zeros((1, 1, S, L), dtype=torch.uint8, device="cuda")
    pv = torch.zeros_like(pk)
    say("single_head encode")
    nk.encode(P, lay, dev(kc[None, :, None, :], torch.float32), dev(vc[None, :, None, :], torch.float32),
              dev([0], torch.int32), pk, pv)
    torch.cuda.synchronize()
    ck, gk, cv, gv = ocodec.encode_tokens(kc, vc, hp)
    compare_codes(pk.cpu().numpy()[0, 0], ck, gk, "single_head K")
    compare_codes(pv.cpu().numpy()[0, 0], cv, gv, "single_head V")

    q = synth.decode_queries(wl, 0)
    scale = 1 / np.sqrt(wl.head_dim)
    ref = oatt.decode_rows(q[0], ck, cv, hp, scale)
    # identical inputs: the oracle's codes
    pk.copy_(dev(ck[None, None], torch.uint8))
    pv.copy_(dev(cv[None, None], torch.uint8))
    say("single_head decode")
    out = nk.decode_attn(P, lay, dev(q, torch.float32), pk, pv, dev([S], torch.int32), S)
    assert_outputs_close(out.cpu().numpy()[0], ref, what="single_head decode")


# ------------------------------------------------ qwen-shaped, moderate size

@pytest.fixture(scope="module")
def qwen_small(nk):
    wl = synth.get_workload("qwen3_8b")
    params = calibrated_params(wl, 0)
    return wl, params, upload_params(nk, params)


@pytest.mark.parametrize("paged", [False, True])
def test_qwen_shape_encode_ragged(nk, qwen_small, paged):
    """32q/8kv, D=128, bf16: GPU encode of 3 sequences x 1100 tokens (ragged tile tail)."""
    wl, params, P = qwen_small
    B, n_new, start = 3, 1100, 37
    cap = 1280
    L, H = wl.groups, wl.num_kv_heads
    if paged:
        bs, bps = 16, cap // 16
        table = np.random.default_rng(7).permutation(B * bps).astype(np.int32).reshape(B, bps)
        lay = nk.CacheLayout(bs, bps, dev(table, torch.int32))
    else:
        bs, bps, table = cap, 1, None
        lay = nk.CacheLayout.contiguous(cap)
    kk = np.empty((B, n_new, H, wl.head_dim))
    vv = np.empty_like(kk)
    for b in range(B):
        for kv in range(H):
            kk[b, :, kv], vv[b, :, kv] = synth.cache_tokens(wl, 0, kv, b, n_new)
    nblocks = B * bps
    pk = torch.zeros((nblocks, H, bs, L), dtype=torch.uint8, device="cuda")
    pv = torch.zeros_like(pk)
    say(f"qwen encode paged={paged}")
    nk.encode(P, lay, dev(kk, torch.bfloat16), dev(vv, torch.bfloat16),
              dev([start] * B, torch.int32), pk, pv)
    torch.cuda.synchronize()
    hk = pk.cpu().numpy().reshape(-1)
    hv = pv.cpu().numpy().reshape(-1)
    lk = lay_kwargs(H, bs, bps, table)
    for b in range(B):
        for kv in range(H):
            ck, gk, cv, gv = ocodec.encode_tokens(kk[b, :, kv], vv[b, :, kv], oatt.head_params(params, kv))
            compare_codes(read_rows(hk, b, kv, start, n_new, groups=L, **lk), ck, gk, f"b{b} kv{kv} K")
            compare_codes(read_rows(hv, b, kv, start, n_new, groups=L, **lk), cv, gv, f"b{b} kv{kv} V")
    # nothing outside the written range was touched
    before = read_rows(hk, 0, 0, 0, start, groups=L, **lk)
    assert not before.any()


def _random_pools(wl, layer, B, cap, H, L):
    ck = synth.random_codes(wl, layer, "k", (B, H, cap, L))
    cv = synth.random_codes(wl, layer, "v", (B, H, cap, L))
    return ck, cv


@pytest.mark.parametrize("window,use_sink", [(0, False), (0, True), (300, True), (1, False)])
def test_qwen_shape_decode_ragged(nk, qwen_small, window, use_sink):
    """Ragged lengths incl. 0 and 1, windows, sinks; every row checked."""
    wl, params, P = qwen_small
    B, cap = 6, 2304
    H, L, G = wl.num_kv_heads, wl.groups, wl.gqa
    lens = np.array([0, 1, 255, 1023, 2000, 2304], dtype=np.int32)
    ck, cv = _random_pools(wl, 0, B, cap, H, L)
    q = synth.decode_queries(wl, 0, batch=B)
    sinks = np.random.default_rng(3).standard_normal(wl.num_q_heads).astype(np.float32) if use_sink else None
    lay = nk.CacheLayout.contiguous(cap)
    say(f"qwen decode window={window} sink={use_sink}")
    out = nk.decode_attn(P, lay, dev(q, torch.bfloat16), dev(ck, torch.uint8), dev(cv, torch.uint8),
                         dev(lens, torch.int32), cap, window=window,
                         sinks=dev(sinks, torch.float32) if use_sink else None).cpu().numpy()
    scale = 1 / np.sqrt(wl.head_dim)
    lk = lay_kwargs(H, cap, 1)
    hk, hv = ck.reshape(-1), cv.reshape(-1)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        for kv in range(H):
            ref[b, kv * G:(kv + 1) * G] = oracle_rows(q, hk, hv, params, b, kv, int(lens[b]), scale, lk,
                                                       window, sinks, G)
    if not use_sink:
        assert np.all(out[0] == 0)            # empty sequence, no sink: zeros
    assert_outputs_close(out.reshape(-1, wl.head_dim), ref.reshape(-1, wl.head_dim),
                         what=f"qwen ragged window={window} sink={use_sink}")


def test_paged_equals_contiguous_and_split_invariance(nk, qwen_small):
    wl, params, P = qwen_small
    B, cap = 2, 4096
    H, L = wl.num_kv_heads, wl.groups
    ck, cv = _random_pools(wl, 0, B, cap, H, L)
    q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
    lens = dev([4096, 3001], torch.int32)
    say("contiguous vs paged")
    out_c = nk.decode_attn(P, nk.CacheLayout.contiguous(cap), q, dev(ck, torch.uint8),
                           dev(cv, torch.uint8), lens, cap)
    bs, bps = 16, cap // 16
    table = np.random.default_rng(11).permutation(B * bps).astype(np.int32).reshape(B, bps)
    flat_k = np.zeros(B * bps * H * bs * L, dtype=np.uint8)
    flat_v = np.zeros_like(flat_k)
    lk = lay_kwargs(H, bs, bps, table)
    for b in range(B):
        for kv in range(H):
            write_rows(flat_k, ck[b, kv], b, kv, 0, **lk)
            write_rows(flat_v, cv[b, kv], b, kv, 0, **lk)
    out_p = nk.decode_attn(P, nk.CacheLayout(bs, bps, dev(table, torch.int32)), q,
                           dev(flat_k, torch.uint8), dev(flat_v, torch.uint8), lens, cap)
    assert torch.equal(out_c, out_p)
    # a larger max_seq_len changes the split plan, not the result (beyond rounding)
    big = torch.zeros((B, H, 8192, L), dtype=torch.uint8, device="cuda")
    big[:, :, :cap] = dev(ck, torch.uint8)
    bigv = torch.zeros_like(big)
    bigv[:, :, :cap] = dev(cv, torch.uint8)
    out_b = nk.decode_attn(P, nk.CacheLayout.contiguous(8192), q, big, bigv, lens, 8192)
    torch.testing.assert_close(out_b, out_c, rtol=1e-5, atol=1e-6)


# ------------------------------------------ GPT-OSS-shaped (D=64, 8 heads/KV)

@pytest.fixture(scope="module")
def gptoss_small(nk):
    wl = synth.get_workload("gptoss_pair")
    params = calibrated_params(wl, 0)
    return wl, params, upload_params(nk, params)


@pytest.mark.parametrize("window,use_sink", [(0, True), (128, True), (1, False), (0, False)])
def test_gptoss_shape_decode_ragged(nk, gptoss_small, window, use_sink):
    """64q/8kv, D=64: ragged lengths incl. 0, 1 and a partial round; windows, sinks; every row."""
    wl, params, P = gptoss_small
    B, cap = 5, 1536
    H, L, G = wl.num_kv_heads, wl.groups, wl.gqa
    lens = np.array([0, 1, 130, 1001, 1536], dtype=np.int32)
    ck, cv = _random_pools(wl, 0, B, cap, H, L)
    q = synth.decode_queries(wl, 0, batch=B)
    sinks = synth.sink_logits(wl, 0) if use_sink else None
    lay = nk.CacheLayout.contiguous(cap)
    say(f"gptoss decode window={window} sink={use_sink}")
    out = nk.decode_attn(P, lay, dev(q, torch.bfloat16), dev(ck, torch.uint8), dev(cv, torch.uint8),
                         dev(lens, torch.int32), cap, window=window,
                         sinks=dev(sinks, torch.float32) if use_sink else None).cpu().numpy()
    scale = 1 / np.sqrt(wl.head_dim)
    lk = lay_kwargs(H, cap, 1)
    hk, hv = ck.reshape(-1), cv.reshape(-1)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        for kv in range(H):
            ref[b, kv * G:(kv + 1) * G] = oracle_rows(q, hk, hv, params, b, kv, int(lens[b]), scale, lk,
                                                       window, sinks, G)
    if not use_sink:
        assert np.all(out[0] == 0)
    assert_outputs_close(out.reshape(-1, wl.head_dim), ref.reshape(-1, wl.head_dim),
                         what=f"gptoss ragged window={window} sink={use_sink}")


def test_gptoss_shape_paged_equals_contiguous(nk, gptoss_small):
    wl, params, P = gptoss_small
    B, cap = 2, 2048
    H, L = wl.num_kv_heads, wl.groups
    ck, cv = _random_pools(wl, 0, B, cap, H, L)
    q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
    lens = dev([2048, 1203], torch.int32)
    sinks = dev(synth.sink_logits(wl, 0), torch.float32)
    say("gptoss contiguous vs paged")
    out_c = nk.decode_attn(P, nk.CacheLayout.contiguous(cap), q, dev(ck, torch.uint8),
                           dev(cv, torch.uint8), lens, cap, sinks=sinks)
    bs, bps = 16, cap // 16
    table = np.random.default_rng(5).permutation(B * bps).astype(np.int32).reshape(B, bps)
    flat_k = np.zeros(B * bps * H * bs * L, dtype=np.uint8)
    flat_v = np.zeros_like(flat_k)
    lk = lay_kwargs(H, bs, bps, table)
    for b in range(B):
        for kv in range(H):
            write_rows(flat_k, ck[b, kv], b, kv, 0, **lk)
            write_rows(flat_v, cv[b, kv], b, kv, 0, **lk)
    out_p = nk.decode_attn(P, nk.CacheLayout(bs, bps, dev(table, torch.int32)), q,
                           dev(flat_k, torch.uint8), dev(flat_v, torch.uint8), lens, cap, sinks=sinks)
    assert torch.equal(out_c, out_p)


# ------------------------------------------- D=64 encoder, head subsets, generic path

@pytest.mark.parametrize("n_new", [1, 3, 101])
def test_gptoss_shape_encode(nk, gptoss_small, n_new):
    """D=64 encode: 1 and 3 tokens (per-token kernel) and 101 tokens (tiled kernel, ragged tail)."""
    wl, params, P = gptoss_small
    B, cap, H, L, D = 3, 256, wl.num_kv_heads, wl.groups, wl.head_dim
    starts = [0, 17, cap - n_new]
    kk = np.empty((B, n_new, H, D))
    vv = np.empty_like(kk)
    for b in range(B):
        for kv in range(H):
            kk[b, :, kv], vv[b, :, kv] = synth.cache_tokens(wl, 0, kv, b, n_new, start=starts[b])
    pk = torch.zeros((B, H, cap, L), dtype=torch.uint8, device="cuda")
    pv = torch.zeros_like(pk)
    say(f"gptoss encode n_new={n_new}")
    nk.encode(P, nk.CacheLayout.contiguous(cap), dev(kk, torch.bfloat16), dev(vv, torch.bfloat16),
              dev(starts, torch.int32), pk, pv)
    torch.cuda.synchronize()
    hk, hv = pk.cpu().numpy(), pv.cpu().numpy()
    for b in range(B):
        s0 = starts[b]
        for kv in range(H):
            ck, gk, cv, gv = ocodec.encode_tokens(kk[b, :, kv], vv[b, :, kv], oatt.head_params(params, kv))
            compare_codes(hk[b, kv, s0:s0 + n_new], ck, gk, f"gptoss b{b} kv{kv} K")
            compare_codes(hv[b, kv, s0:s0 + n_new], cv, gv, f"gptoss b{b} kv{kv} V")
        # rows outside [start, start + n_new) stay untouched
        assert not hk[b, :, :s0].any() and not hk[b, :, s0 + n_new:].any()
        assert not hv[b, :, :s0].any() and not hv[b, :, s0 + n_new:].any()


def _head_subset(x, hkv, gqa_full, gqa):
    """Keep the first ``gqa`` query heads of each KV head: [B][Hkv*gqa_full][...] -> [B][Hkv*gqa][...]."""
    shp = x.shape
    y = x.reshape(shp[0], hkv, gqa_full, *shp[2:])[:, :, :gqa]
    return np.ascontiguousarray(y.reshape(shp[0], hkv * gqa, *shp[2:]))


@pytest.mark.parametrize("shape,gqa", [("gptoss_pair", 1), ("gptoss_pair", 4), ("qwen3_8b", 1),
                                       ("qwen3_8b", 2)])
def test_fewer_query_heads_per_kv_head(nk, shape, gqa):
    """Table kernels with fewer query heads per KV head than their head slots (D=64 and D=128)."""
    wl = synth.get_workload(shape)
    params = calibrated_params(wl, 0)
    P = upload_params(nk, params)
    B, cap = 3, 1200
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    lens = np.array([1200, 77, 640], dtype=np.int32)
    ck, cv = _random_pools(wl, 0, B, cap, H, L)
    q = _head_subset(synth.decode_queries(wl, 0, batch=B), H, wl.gqa, gqa)
    rng = np.random.default_rng(29)
    sinks = rng.standard_normal(H * gqa).astype(np.float32)
    say(f"{shape} decode with {gqa} query heads per KV head")
    out = nk.decode_attn(P, nk.CacheLayout.contiguous(cap), dev(q, torch.bfloat16), dev(ck, torch.uint8),
                         dev(cv, torch.uint8), dev(lens, torch.int32), cap,
                         sinks=dev(sinks, torch.float32)).cpu().numpy()
    scale = 1 / np.sqrt(D)
    lk = lay_kwargs(H, cap, 1)
    hk, hv = ck.reshape(-1), cv.reshape(-1)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        for kv in range(H):
            ref[b, kv * gqa:(kv + 1) * gqa] = oracle_rows(q, hk, hv, params, b, kv, int(lens[b]), scale,
                                                           lk, 0, sinks, gqa)
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D), what=f"{shape} gqa={gqa}")


@pytest.mark.parametrize("window,use_sink", [(0, False), (200, True)])
def test_generic_path_paged_block8(nk, qwen_small, window, use_sink):
    """Pages of 8 tokens are outside the table kernels' layout: the split-K kernels take them."""
    wl, params, P = qwen_small
    B, cap, bs = 4, 1000, 8
    bps = cap // bs
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    lens = np.array([0, 9, 517, 1000], dtype=np.int32)
    ck, cv = _random_pools(wl, 0, B, cap, H, L)
    table = np.random.default_rng(13).permutation(B * bps).astype(np.int32).reshape(B, bps)
    lk = lay_kwargs(H, bs, bps, table)
    flat_k = np.zeros(B * bps * H * bs * L, dtype=np.uint8)
    flat_v = np.zeros_like(flat_k)
    for b in range(B):
        for kv in range(H):
            write_rows(flat_k, ck[b, kv], b, kv, 0, **lk)
            write_rows(flat_v, cv[b, kv], b, kv, 0, **lk)
    q = synth.decode_queries(wl, 0, batch=B)
    sinks = np.random.default_rng(31).standard_normal(wl.num_q_heads).astype(np.float32) if use_sink else None
    say(f"generic path block_size=8 window={window} sink={use_sink}")
    out = nk.decode_attn(P, nk.CacheLayout(bs, bps, dev(table, torch.int32)), dev(q, torch.bfloat16),
                         dev(flat_k, torch.uint8), dev(flat_v, torch.uint8), dev(lens, torch.int32), cap,
                         window=window, sinks=dev(sinks, torch.float32) if use_sink else None).cpu().numpy()
    scale = 1 / np.sqrt(D)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        for kv in range(H):
            ref[b, kv * G:(kv + 1) * G] = oracle_rows(q, flat_k, flat_v, params, b, kv, int(lens[b]), scale,
                                                       lk, window, sinks, G)
    if not use_sink:
        assert np.all(out[0] == 0)
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D),
                         what=f"generic block8 window={window} sink={use_sink}")


# ----------------------------------------- fused step: append the token, then decode

def _step_inputs(wl, B, cap, lens, seed_layer=0):
    """History codes for positions < lens[b] - 1 and the step's token at lens[b] - 1."""
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    ck, cv = _random_pools(wl, seed_layer, B, cap, H, L)
    kn = np.empty((B, H, D))
    vn = np.empty_like(kn)
    for b in range(B):
        for kv in range(H):
            kn[b, kv], vn[b, kv] = (x[0] for x in synth.cache_tokens(wl, seed_layer, kv, b, 1,
                                                                       start=max(int(lens[b]) - 1, 0)))
    return ck, cv, kn, vn


@pytest.mark.parametrize("paged,window,use_sink", [(False, 0, True), (False, 300, True), (True, 0, False),
                                                   (False, 1, False)])
def test_append_decode_matches_oracle(nk, qwen_small, paged, window, use_sink):
    """One-launch step at the Qwen shape: the token's codes bit-exact, the output within tolerance."""
    wl, params, P = qwen_small
    B, cap = 6, 2304
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    lens = np.array([1, 2, 65, 1024, 2000, 2304], dtype=np.int32)
    ck, cv, kn, vn = _step_inputs(wl, B, cap, lens)
    if paged:
        bs, bps = 16, cap // 16
        table = np.random.default_rng(17).permutation(B * bps).astype(np.int32).reshape(B, bps)
        lay = nk.CacheLayout(bs, bps, dev(table, torch.int32))
    else:
        bs, bps, table = cap, 1, None
        lay = nk.CacheLayout.contiguous(cap)
    lk = lay_kwargs(H, bs, bps, table)
    flat_k = np.zeros(B * bps * H * bs * L, dtype=np.uint8)
    flat_v = np.zeros_like(flat_k)
    for b in range(B):
        for kv in range(H):
            write_rows(flat_k, ck[b, kv], b, kv, 0, **lk)
            write_rows(flat_v, cv[b, kv], b, kv, 0, **lk)
    pk, pv = dev(flat_k, torch.uint8), dev(flat_v, torch.uint8)
    q = synth.decode_queries(wl, 0, batch=B)
    sinks = np.random.default_rng(5).standard_normal(wl.num_q_heads).astype(np.float32) if use_sink else None
    say(f"append+decode paged={paged} window={window} sink={use_sink}")
    out = nk.append_decode_attn(P, lay, dev(kn, torch.bfloat16), dev(vn, torch.bfloat16), dev(q, torch.bfloat16),
                                pk, pv, dev(lens, torch.int32), cap, window=window,
                                sinks=dev(sinks, torch.float32) if use_sink else None).cpu().numpy()
    hk, hv = pk.cpu().numpy(), pv.cpu().numpy()
    ref_k, ref_v = flat_k.copy(), flat_v.copy()
    for b in range(B):
        p = int(lens[b]) - 1
        for kv in range(H):
            okk, ogk, ovv, ogv = ocodec.encode_tokens(kn[b, kv][None], vn[b, kv][None], oatt.head_params(params, kv))
            compare_codes(read_rows(hk, b, kv, p, 1, groups=L, **lk), okk, ogk, f"step b{b} kv{kv} K")
            compare_codes(read_rows(hv, b, kv, p, 1, groups=L, **lk), ovv, ogv, f"step b{b} kv{kv} V")
            write_rows(ref_k, okk, b, kv, p, **lk)
            write_rows(ref_v, ovv, b, kv, p, **lk)
            # every other row untouched
        before = read_rows(hk, b, 0, 0, p, groups=L, **lk)
        assert np.array_equal(before, read_rows(flat_k, b, 0, 0, p, groups=L, **lk))
    scale = 1 / np.sqrt(D)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        for kv in range(H):
            ref[b, kv * G:(kv + 1) * G] = oracle_rows(q, ref_k, ref_v, params, b, kv, int(lens[b]), scale, lk,
                                                       window, sinks, G)
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D),
                         what=f"append+decode paged={paged} window={window} sink={use_sink}")


@pytest.mark.parametrize("fused,window", [(False, 0), (False, 5000), (True, 0), (True, 5000)])
@pytest.mark.parametrize("hkv", [8, 2])
def test_many_splits(nk, qwen_small, fused, window, hkv):
    """Two sequences at a long cap, one of them short.  Eight KV heads at
    16384 tokens: 16 splits per KV head, one combine.  Two KV heads at 32768
    tokens: 64 splits, combined in groups of splits first; the short
    sequence leaves whole groups without tokens."""
    wl0, params0, _ = qwen_small
    wl = wl0.scaled(num_kv_heads=hkv, num_q_heads=hkv * wl0.gqa)
    params = {k: v[:hkv] for k, v in params0.items()}
    P = upload_params(nk, params)
    B, cap = 2, (16384 if hkv == 8 else 32768)
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    lens = np.array([cap, 700], dtype=np.int32)
    ck, cv, kn, vn = _step_inputs(wl, B, cap, lens)
    q = synth.decode_queries(wl, 0, batch=B)
    sinks = np.random.default_rng(21).standard_normal(wl.num_q_heads).astype(np.float32)
    lay = nk.CacheLayout.contiguous(cap)
    pk, pv = dev(ck, torch.uint8), dev(cv, torch.uint8)
    args = dict(window=window, sinks=dev(sinks, torch.float32))
    say(f"many splits hkv={hkv} fused={fused} window={window}")
    if fused:
        out = nk.append_decode_attn(P, lay, dev(kn, torch.bfloat16), dev(vn, torch.bfloat16),
                                    dev(q, torch.bfloat16), pk, pv, dev(lens, torch.int32), cap, **args)
    else:
        out = nk.decode_attn(P, lay, dev(q, torch.bfloat16), pk, pv, dev(lens, torch.int32), cap, **args)
    out = out.cpu().numpy()
    ref_k, ref_v = ck.copy(), cv.copy()
    if fused:
        for b in range(B):
            p = int(lens[b]) - 1
            for kv in range(H):
                okk, _, ovv, _ = ocodec.encode_tokens(kn[b, kv][None], vn[b, kv][None], oatt.head_params(params, kv))
                ref_k[b, kv, p], ref_v[b, kv, p] = okk[0], ovv[0]
    lk = lay_kwargs(H, cap, 1)
    hk, hv = ref_k.reshape(-1), ref_v.reshape(-1)
    scale = 1 / np.sqrt(D)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        for kv in range(H):
            ref[b, kv * G:(kv + 1) * G] = oracle_rows(q, hk, hv, params, b, kv, int(lens[b]), scale, lk,
                                                       window, sinks, G)
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D),
                         what=f"many splits hkv={hkv} fused={fused} window={window}")


@pytest.mark.parametrize("shape", ["qwen3_8b", "gptoss_pair"])
def test_append_decode_equals_encode_then_decode(nk, shape):
    """The step in one call stores the same bytes as the one-token encode and gives the decode's output."""
    wl = synth.get_workload(shape)
    params = calibrated_params(wl, 0)
    P = upload_params(nk, params)
    B, cap = 4, 4096
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    lens = np.array([4096, 3001, 64, 1], dtype=np.int32)
    ck, cv, kn, vn = _step_inputs(wl, B, cap, lens)
    q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
    sinks = dev(synth.sink_logits(wl, 0), torch.float32) if wl.sinks else None
    lay = nk.CacheLayout.contiguous(cap)
    lens_d = dev(lens, torch.int32)
    kn_d, vn_d = dev(kn, torch.bfloat16), dev(vn, torch.bfloat16)
    say(f"{shape}: two calls")
    pk1, pv1 = dev(ck, torch.uint8), dev(cv, torch.uint8)
    nk.encode(P, lay, kn_d[:, None], vn_d[:, None], lens_d - 1, pk1, pv1)
    out1 = nk.decode_attn(P, lay, q, pk1, pv1, lens_d, cap, sinks=sinks)
    say(f"{shape}: one call")
    pk2, pv2 = dev(ck, torch.uint8), dev(cv, torch.uint8)
    out2 = nk.append_decode_attn(P, lay, kn_d, vn_d, q, pk2, pv2, lens_d, cap, sinks=sinks)
    torch.cuda.synchronize()
    assert torch.equal(pk1, pk2) and torch.equal(pv1, pv2)
    # Inside a split the new token's probability passes through the fp16 value
    # operand (relative rounding 2^-12 of its weight); the one-call step adds
    # its term in fp32 after the combine.  The two differ by that rounding.
    err = (out2 - out1).abs().amax(dim=-1) / out1.norm(dim=-1).clamp_min(1e-30)
    print(f"[parity] {shape} one-call vs two-call worst_rel_diff={float(err.max()):.3e}", flush=True)
    assert float(err.max()) <= 1e-4


def test_shared_workspace_across_shapes(nk, qwen_small):
    """One workspace serves calls of different shapes and split counts in turn.

    The splits of a (sequence, KV head) exchange tagged words in the workspace
    and the combining split empties what it read; a word left behind by an
    earlier call of another shape must never be taken for a partial.  Each
    call is compared with the same call on a fresh workspace."""
    wl, params, P = qwen_small
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    cases = [(4, 4096, [4096, 3001, 64, 1], 0), (2, 8192, [8192, 5000], 0), (4, 4096, [4096, 3001, 64, 1], 300),
             (1, 16384, [16000], 0), (8, 2048, [2048, 2047, 1000, 64, 63, 1, 2, 1500], 0)]
    inputs = []
    for B, cap, lens, window in cases:
        lens = np.array(lens, dtype=np.int32)
        ck, cv, kn, vn = _step_inputs(wl, B, cap, lens)
        q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
        inputs.append((B, cap, lens, window, ck, cv, dev(kn, torch.bfloat16), dev(vn, torch.bfloat16), q))
    need = max(nk.decode_workspace_bytes(P, B, wl.num_q_heads, cap) for B, cap, *_ in inputs)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for rep in range(2):
        for i, (B, cap, lens, window, ck, cv, kn, vn, q) in enumerate(inputs):
            lay = nk.CacheLayout.contiguous(cap)
            lens_d = dev(lens, torch.int32)
            for fused in (False, True):
                say(f"shared workspace rep={rep} case={i} fused={fused}")
                outs = []
                for w in (ws, None):
                    pk, pv = dev(ck, torch.uint8), dev(cv, torch.uint8)
                    if fused:
                        outs.append(nk.append_decode_attn(P, lay, kn, vn, q, pk, pv, lens_d, cap, window=window,
                                                          workspace=w))
                    else:
                        outs.append(nk.decode_attn(P, lay, q, pk, pv, lens_d, cap, window=window, workspace=w))
                torch.cuda.synchronize()
                err = (outs[0] - outs[1]).abs().amax(dim=-1) / outs[1].norm(dim=-1).clamp_min(1e-30)
                assert torch.isfinite(outs[0]).all()
                assert float(err.max()) <= 1e-4, (rep, i, fused, float(err.max()))


def test_side_stream_temporaries(nk, qwen_small):
    """Calls on a stream other than torch's current one, with the output and
    the zeroed workspace left to the binding: those are created and filled on
    the call's stream, so the kernel sees a filled workspace and the memory
    is not handed to other streams' work while the kernel runs.  The default
    stream meanwhile allocates and fills memory of the workspace's size; the
    results must equal the same calls on the default stream."""
    wl, params, P = qwen_small
    B, cap = 4, 4096
    lens = np.array([4096, 3001, 64, 1], dtype=np.int32)
    ck, cv, kn, vn = _step_inputs(wl, B, cap, lens)
    q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
    kn_d, vn_d = dev(kn, torch.bfloat16), dev(vn, torch.bfloat16)
    lay = nk.CacheLayout.contiguous(cap)
    lens_d = dev(lens, torch.int32)
    need = nk.decode_workspace_bytes(P, B, wl.num_q_heads, cap)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    for fused in (False, True):
        say(f"side stream fused={fused}: default-stream reference")
        pk, pv = dev(ck, torch.uint8), dev(cv, torch.uint8)
        if fused:
            ref = nk.append_decode_attn(P, lay, kn_d, vn_d, q, pk, pv, lens_d, cap)
        else:
            ref = nk.decode_attn(P, lay, q, pk, pv, lens_d, cap)
        torch.cuda.synchronize()
        for rep in range(3):
            say(f"side stream fused={fused} rep={rep}")
            pk, pv = dev(ck, torch.uint8), dev(cv, torch.uint8)
            side.wait_stream(main)  # the inputs were written on the default stream
            if fused:
                out = nk.append_decode_attn(P, lay, kn_d, vn_d, q, pk, pv, lens_d, cap, stream=side)
            else:
                out = nk.decode_attn(P, lay, q, pk, pv, lens_d, cap, stream=side)
            junk = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda")  # default-stream allocation
            main.wait_stream(side)
            torch.cuda.synchronize()
            del junk
            assert torch.isfinite(out).all()
            err = (out - ref).abs().amax(dim=-1) / ref.norm(dim=-1).clamp_min(1e-30)
            assert float(err.max()) <= 1e-4, (fused, rep, float(err.max()))


# ------------------------------------------------- full-size configurations

def _full_decode(nk, wl, layer, params, units, window=0, batch=None, cap=None):
    B = wl.batch if batch is None else batch
    cap = wl.seq_len if cap is None else cap
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    P = upload_params(nk, params)
    ck, cv = _random_pools(wl, layer, B, cap, H, L)
    q = synth.decode_queries(wl, layer, batch=B)
    sinks = synth.sink_logits(wl, layer)
    lens = np.full(B, cap, dtype=np.int32)
    say(f"{wl.name} layer {layer} full decode B={B} S={cap} window={window}")
    out = nk.decode_attn(P, nk.CacheLayout.contiguous(cap), dev(q, qdtype(wl)), dev(ck, torch.uint8),
                         dev(cv, torch.uint8), dev(lens, torch.int32), cap, window=window,
                         sinks=dev(sinks, torch.float32) if sinks is not None else None)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    scale = 1 / np.sqrt(D)
    lk = lay_kwargs(H, cap, 1)
    hk, hv = ck.reshape(-1), cv.reshape(-1)
    gots, refs = [], []
    for b, kv in units:
        refs.append(oracle_rows(q, hk, hv, params, b, kv, cap, scale, lk, window, sinks, G))
        gots.append(out[b, kv * G:(kv + 1) * G])
    assert_outputs_close(np.concatenate(gots), np.concatenate(refs), what=f"{wl.name} L{layer}")
    assert np.isfinite(out).all()


def test_qwen3_8b_full_decode(nk):
    wl = synth.get_workload("qwen3_8b")
    _full_decode(nk, wl, 0, calibrated_params(wl, 0), [(0, 0), (3, 5), (7, 7)])


def test_sweep_b64_s32k_decode(nk):
    wl = synth.get_workload("sweep_b64_s32k")
    _full_decode(nk, wl, 0, calibrated_params(synth.get_workload("qwen3_8b"), 0),
                 [(0, 1), (40, 3), (63, 6)])


def test_sweep_b1_s128k_decode(nk):
    wl = synth.get_workload("sweep_b1_s128k")
    _full_decode(nk, wl, 0, calibrated_params(synth.get_workload("qwen3_8b"), 0), [(0, 0), (0, 4)])


@pytest.mark.parametrize("layer", [0, 1])
def test_gptoss_pair_decode(nk, layer):
    wl = synth.get_workload("gptoss_pair")
    _full_decode(nk, wl, layer, calibrated_params(wl, layer), [(0, 0), (9, 2), (15, 7)],
                 window=wl.windows[layer])


def _device_tokens(wl, batch, n, start):
    """Seeded device-side keys and values [B][n][Hkv][D] (bf16) of every sequence."""
    kk = torch.empty((batch, n, wl.num_kv_heads, wl.head_dim), dtype=torch.bfloat16, device="cuda")
    vv = torch.empty_like(kk)
    for b in range(batch):
        kk[b], vv[b] = synth.device_cache_tokens(wl, 0, b, n, start, "cuda")
    return kk, vv


def _pool_rows(pool_host, b_list, kv, start, n, *, hkv, groups, block_size, blocks_per_seq, table=None):
    """Code rows of positions [start, start+n) of sequences b_list, KV head kv, stacked."""
    offs = np.concatenate([pool_offsets(b, kv, np.arange(start, start + n), hkv=hkv, groups=groups,
                                        block_size=block_size, blocks_per_seq=blocks_per_seq, table=table)
                           for b in b_list])
    return pool_host[offs[:, None] + np.arange(groups)[None, :]]


def _check_all_codes(params, kk, vv, pk_host, pv_host, start, lay, what):
    """Every code of the tokens kk, vv [B][n][Hkv][D] against the oracle, one KV head at a time.

    Returns the oracle's codes {kv: (ck [B*n][L], cv)} (sequence-major rows)."""
    B, n, H, D = kk.shape
    L = D // 4
    kh = kk.float().cpu().numpy()
    vh = vv.float().cpu().numpy()
    codes = {}
    for kv in range(H):
        K = kh[:, :, kv].reshape(-1, D).astype(np.float64)
        V = vh[:, :, kv].reshape(-1, D).astype(np.float64)
        ck, gk, cv, gv = ocodec.encode_tokens(K, V, oatt.head_params(params, kv))
        compare_codes(_pool_rows(pk_host, range(B), kv, start, n, groups=L, **lay), ck, gk,
                      f"{what} kv{kv} K ({B} sequences x {n})")
        compare_codes(_pool_rows(pv_host, range(B), kv, start, n, groups=L, **lay), cv, gv,
                      f"{what} kv{kv} V ({B} sequences x {n})")
        codes[kv] = (ck, cv)
    return codes


def test_qwen3_8b_full_encode(nk):
    """Full-size GPU encode of B=8 x 8 KV heads x 16384 tokens (one bulk call); every code against the oracle."""
    wl = synth.get_workload("qwen3_8b")
    params = calibrated_params(wl, 0)
    P = upload_params(nk, params)
    B, S, H, L = wl.batch, wl.seq_len, wl.num_kv_heads, wl.groups
    kk, vv = _device_tokens(wl, B, S, 0)
    pk = torch.zeros((B, H, S, L), dtype=torch.uint8, device="cuda")
    pv = torch.zeros_like(pk)
    say("qwen3_8b full encode")
    nk.encode(P, nk.CacheLayout.contiguous(S), kk, vv, torch.zeros(B, dtype=torch.int32, device="cuda"), pk, pv)
    torch.cuda.synchronize()
    _check_all_codes(params, kk, vv, pk.cpu().numpy().reshape(-1), pv.cpu().numpy().reshape(-1), 0,
                     lay_kwargs(H, S, 1), "qwen3_8b encode")


@pytest.mark.parametrize("lens", ["full", "ragged"])
def test_step_at_qwen3_8b_bench_shape(nk, lens):
    """The benchmarked call at its shape: nova_kv_append_decode_attn at B=8, S=16384,
    32 q / 8 KV heads (one launch, four splits per (sequence, KV head), the new
    token's encode shared by them).  The appended codes of all 64 units are
    checked bit-exact, every other row of the pools unchanged, and 8 sampled
    (sequence, KV head) units' outputs against the oracle over the history
    codes and the oracle's own codes of the new token.  "ragged" gives the
    sequences lengths from 16384 down to 1 at the same max_seq_len, so the
    new token's items fall to 1..4 splits."""
    wl = synth.get_workload("qwen3_8b")
    params = calibrated_params(wl, 0)
    P = upload_params(nk, params)
    B, S, H, L, G, D = wl.batch, wl.seq_len, wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    seq = np.full(B, S, dtype=np.int32) if lens == "full" else \
        np.array([16384, 16000, 12289, 8193, 4097, 4096, 100, 1], dtype=np.int32)
    ck, cv, kn, vn = _step_inputs(wl, B, S, seq)
    q = synth.decode_queries(wl, 0)
    pk, pv = dev(ck, torch.uint8), dev(cv, torch.uint8)
    before_k, before_v = pk.clone(), pv.clone()
    say(f"bench-shape step lens={lens}")
    out = nk.append_decode_attn(P, nk.CacheLayout.contiguous(S), dev(kn, torch.bfloat16), dev(vn, torch.bfloat16),
                                dev(q, torch.bfloat16), pk, pv, dev(seq, torch.int32), S)
    torch.cuda.synchronize()
    # every row but the new token's unchanged
    mask = torch.ones((B, 1, S, 1), dtype=torch.bool, device="cuda")
    for b in range(B):
        mask[b, 0, seq[b] - 1] = False
    assert torch.equal(pk.masked_select(mask.expand_as(pk)), before_k.masked_select(mask.expand_as(pk)))
    assert torch.equal(pv.masked_select(mask.expand_as(pv)), before_v.masked_select(mask.expand_as(pv)))
    hk, hv = pk.cpu().numpy(), pv.cpu().numpy()
    ref_k, ref_v = ck.copy(), cv.copy()
    new_k, new_v, gap_k, gap_v = [], [], [], []
    for b in range(B):
        p = int(seq[b]) - 1
        for kv in range(H):
            okk, ogk, ovv, ogv = ocodec.encode_tokens(kn[b, kv][None], vn[b, kv][None], oatt.head_params(params, kv))
            new_k.append((hk[b, kv, p], okk[0], ogk[0]))
            new_v.append((hv[b, kv, p], ovv[0], ogv[0]))
            ref_k[b, kv, p], ref_v[b, kv, p] = okk[0], ovv[0]
    for side, rows in (("K", new_k), ("V", new_v)):
        compare_codes(np.stack([r[0] for r in rows]), np.stack([r[1] for r in rows]), np.stack([r[2] for r in rows]),
                      f"bench-shape step lens={lens} new token {side} (64 units)")
    out = out.cpu().numpy()
    scale = 1 / np.sqrt(D)
    units = [(0, 0), (1, 3), (2, 6), (3, 1), (4, 4), (5, 7), (6, 2), (7, 5)]
    gots, refs = [], []
    for b, kv in units:
        hp = oatt.head_params(params, kv)
        n = int(seq[b])
        refs.append(oatt.decode_rows(q[b, kv * G:(kv + 1) * G], ref_k[b, kv, :n], ref_v[b, kv, :n], hp, scale))
        gots.append(out[b, kv * G:(kv + 1) * G])
    assert_outputs_close(np.concatenate(gots), np.concatenate(refs), what=f"bench-shape step lens={lens}")
    assert np.isfinite(out).all()


@pytest.mark.timeout(900)
def test_append_paged_then_decode(nk):
    """The append workload as specified: 32 sequences of a paged cache (16-token
    blocks, shuffled block table) hold a 28,672-token history encoded by the
    same GPU encoder (untimed set-up), then 4096 new tokens per sequence are
    appended in one call and one decode step reads all 32,768 positions.
    Every appended code of all 256 (sequence, KV head) units is checked
    bit-exact; for sampled units the history codes are checked too and the
    decode output is compared with the oracle's decode over its own codes.
    Inputs come from the seeded device-side generator."""
    wl = synth.get_workload("append_paged")
    params = calibrated_params(synth.get_workload("qwen3_8b"), 0)
    P = upload_params(nk, params)
    B, S, H, L, D, G = wl.batch, wl.seq_len, wl.num_kv_heads, wl.groups, wl.head_dim, wl.gqa
    bs = wl.block_size
    bps = S // bs
    start = S - wl.n_new
    table = synth.shuffled_block_table(wl)
    lk = lay_kwargs(H, bs, bps, table)
    lay = nk.CacheLayout(bs, bps, dev(table, torch.int32))
    pk = torch.zeros((B * bps, H, bs, L), dtype=torch.uint8, device="cuda")
    pv = torch.zeros_like(pk)
    say("append_paged: history encode (28672 tokens x 32 sequences)")
    hk, hv = _device_tokens(wl, B, start, 0)
    nk.encode(P, lay, hk, hv, torch.zeros(B, dtype=torch.int32, device="cuda"), pk, pv)
    say("append_paged: append 4096 tokens x 32 sequences")
    kk, vv = _device_tokens(wl, B, wl.n_new, start)
    nk.encode(P, lay, kk, vv, torch.full((B,), start, dtype=torch.int32, device="cuda"), pk, pv)
    torch.cuda.synchronize()
    say("append_paged: oracle check of every appended code")
    gk_pool, gv_pool = pk.cpu().numpy().reshape(-1), pv.cpu().numpy().reshape(-1)
    new_codes = _check_all_codes(params, kk, vv, gk_pool, gv_pool, start, lk, "append")
    del kk, vv
    say("append_paged: decode at 32768")
    q = synth.decode_queries(wl, 0)
    out = nk.decode_attn(P, lay, dev(q, torch.bfloat16), pk, pv, torch.full((B,), S, dtype=torch.int32,
                                                                            device="cuda"), S)
    out = out.cpu().numpy()
    scale = 1 / np.sqrt(D)
    gots, refs = [], []
    for b, kv in [(0, 0), (13, 4), (31, 7)]:
        hp = oatt.head_params(params, kv)
        xk = hk[b, :, kv].float().cpu().numpy().astype(np.float64)
        xv = hv[b, :, kv].float().cpu().numpy().astype(np.float64)
        ck, gk, cv, gv = ocodec.encode_tokens(xk, xv, hp)
        compare_codes(_pool_rows(gk_pool, [b], kv, 0, start, groups=L, **lk), ck, gk, f"append history b{b} kv{kv} K")
        compare_codes(_pool_rows(gv_pool, [b], kv, 0, start, groups=L, **lk), cv, gv, f"append history b{b} kv{kv} V")
        nck, ncv = new_codes[kv]
        rows = slice(b * wl.n_new, (b + 1) * wl.n_new)
        refs.append(oatt.decode_rows(q[b, kv * G:(kv + 1) * G], np.concatenate([ck, nck[rows]]),
                                     np.concatenate([cv, ncv[rows]]), hp, scale))
        gots.append(out[b, kv * G:(kv + 1) * G])
    assert_outputs_close(np.concatenate(gots), np.concatenate(refs), what="append_paged decode")
    assert np.isfinite(out).all()
