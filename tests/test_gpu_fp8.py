"""GPU parity of fp8 E4M3 codebooks (the codebooks snapped to fp8 and stored
as one byte per coordinate).

* Against the fp64 CPU oracle run on the snapped codebooks: codes bit-exact
  except near-ties, decode outputs within 2e-3 of each row's L2 norm, on every
  kernel family and the one-launch step.
* Against the fp16 storage of the same snapped values: every E4M3 value is
  exact in fp16, so the kernels must give identical bits in both formats.
"""

import numpy as np
import pytest
import torch

import synth
from helpers import assert_outputs_close, compare_codes, read_rows
from oracle import attention as oatt
from oracle import codec as ocodec
from oracle import fp8 as ofp8
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


def both_formats(nk, params, key_scale=False):
    """(P8, P16): the snapped codebooks as fp8 bytes and as fp16 values."""
    b8 = dict(params, cb_k=ofp8.e4m3_bits(params["cb_k"].astype(np.float64)),
              cb_v=ofp8.e4m3_bits(params["cb_v"].astype(np.float64)))
    P8 = nk.NovaKVParams.from_arrays(b8, key_scale=key_scale)
    P16 = nk.NovaKVParams.from_arrays(params, key_scale=key_scale)
    assert P8.fp8_codebooks and not P16.fp8_codebooks
    return P8, P16


@pytest.fixture(scope="module")
def qwen8(nk):
    wl = synth.get_workload("qwen3_8b")
    params = calibrated_params(wl, 0, fp8=True)
    return (wl, params) + both_formats(nk, params)


@pytest.fixture(scope="module")
def gptoss8(nk):
    wl = synth.get_workload("gptoss_pair")
    params = calibrated_params(wl, 0, fp8=True)
    return (wl, params) + both_formats(nk, params)


@pytest.mark.parametrize("shape,n_new", [("qwen3_8b", 1100), ("qwen3_8b", 3), ("gptoss_pair", 40),
                                         ("gptoss_pair", 1)])
def test_encode(nk, qwen8, gptoss8, shape, n_new):
    wl, params, P8, P16 = qwen8 if shape == "qwen3_8b" else gptoss8
    B, start, cap = 2, 37, 1280
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    kk = np.empty((B, n_new, H, D))
    vv = np.empty_like(kk)
    for b in range(B):
        for kv in range(H):
            kk[b, :, kv], vv[b, :, kv] = synth.cache_tokens(wl, 0, kv, b, n_new)
    lay = nk.CacheLayout.contiguous(cap)
    pools = []
    for P in (P8, P16):
        pk = torch.zeros((B, H, cap, L), dtype=torch.uint8, device="cuda")
        pv = torch.zeros_like(pk)
        say(f"fp8 encode {shape} n_new={n_new} fp8={P.fp8_codebooks}")
        nk.encode(P, lay, dev(kk, torch.bfloat16), dev(vv, torch.bfloat16), dev([start] * B, torch.int32), pk, pv)
        pools.append((pk, pv))
    torch.cuda.synchronize()
    assert torch.equal(pools[0][0], pools[1][0]) and torch.equal(pools[0][1], pools[1][1])
    hk, hv = pools[0][0].cpu().numpy(), pools[0][1].cpu().numpy()
    for b in range(B):
        for kv in range(H):
            ck, gk, cv, gv = ocodec.encode_tokens(kk[b, :, kv], vv[b, :, kv], oatt.head_params(params, kv))
            compare_codes(hk[b, kv, start:start + n_new], ck, gk, f"{shape} b{b} kv{kv} K")
            compare_codes(hv[b, kv, start:start + n_new], cv, gv, f"{shape} b{b} kv{kv} V")


def _decode_both(nk, wl, params, P8, P16, lens, cap, window=0, sinks=None, paged_bs=None, what=""):
    B = len(lens)
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    ck = synth.random_codes(wl, 0, "k", (B, H, cap, L))
    cv = synth.random_codes(wl, 0, "v", (B, H, cap, L))
    if paged_bs:
        bps = cap // paged_bs
        table = np.random.default_rng(13).permutation(B * bps).astype(np.int32).reshape(B, bps)
        # physical block table[b][i] of the flat pool holds logical block i of sequence b
        flat_k = np.zeros((B * bps, H, paged_bs, L), dtype=np.uint8)
        flat_v = np.zeros_like(flat_k)
        for b in range(B):
            for i in range(bps):
                flat_k[table[b, i]] = ck[b, :, i * paged_bs:(i + 1) * paged_bs]
                flat_v[table[b, i]] = cv[b, :, i * paged_bs:(i + 1) * paged_bs]
        lay = nk.CacheLayout(paged_bs, bps, dev(table, torch.int32))
    else:
        flat_k, flat_v = ck, cv
        lay = nk.CacheLayout.contiguous(cap)
    q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
    outs = []
    for P in (P8, P16):
        say(f"fp8 decode {what} fp8={P.fp8_codebooks}")
        outs.append(nk.decode_attn(P, lay, q, dev(flat_k, torch.uint8), dev(flat_v, torch.uint8),
                                   dev(np.asarray(lens, dtype=np.int32), torch.int32), cap, window=window,
                                   sinks=dev(sinks, torch.float32) if sinks is not None else None))
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1]), f"{what}: fp8 and fp16 storage of the same values differ"
    out = outs[0].cpu().numpy()
    qh = synth.decode_queries(wl, 0, batch=B)
    scale = 1 / np.sqrt(D)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        S = int(lens[b])
        for kv in range(H):
            heads = slice(kv * G, (kv + 1) * G)
            ref[b, heads] = oatt.decode_rows(qh[b, heads], ck[b, kv, :S], cv[b, kv, :S], oatt.head_params(params, kv),
                                             scale, window, None if sinks is None else sinks[heads])
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D), what=f"fp8 {what}")


@pytest.mark.parametrize("window,use_sink,paged", [(0, False, False), (300, True, False), (0, True, True)])
def test_qwen_shape_decode(nk, qwen8, window, use_sink, paged):
    wl, params, P8, P16 = qwen8
    sinks = np.random.default_rng(3).standard_normal(wl.num_q_heads).astype(np.float32) if use_sink else None
    _decode_both(nk, wl, params, P8, P16, [0, 1, 255, 1023, 2000, 2304], 2304, window, sinks,
                 paged_bs=16 if paged else None, what=f"qwen window={window} sink={use_sink} paged={paged}")


@pytest.mark.parametrize("window", [0, 128])
def test_gptoss_shape_decode(nk, gptoss8, window):
    wl, params, P8, P16 = gptoss8
    _decode_both(nk, wl, params, P8, P16, [2048, 1500, 129, 1], 2048, window, synth.sink_logits(wl, 0),
                 what=f"gptoss window={window}")


def test_generic_path_block8_decode(nk, qwen8):
    wl, params, P8, P16 = qwen8
    _decode_both(nk, wl, params, P8, P16, [0, 9, 517, 1000], 1000, 200, None, paged_bs=8, what="block8")


def test_qwen3_8b_full_size_sampled(nk, qwen8):
    wl, params, P8, _ = qwen8
    B, cap = wl.batch, wl.seq_len
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    ck = synth.random_codes(wl, 0, "k", (B, H, cap, L))
    cv = synth.random_codes(wl, 0, "v", (B, H, cap, L))
    q = synth.decode_queries(wl, 0, batch=B)
    say(f"fp8 qwen full decode B={B} S={cap}")
    out = nk.decode_attn(P8, nk.CacheLayout.contiguous(cap), dev(q, torch.bfloat16), dev(ck, torch.uint8),
                         dev(cv, torch.uint8), dev(np.full(B, cap), torch.int32), cap).cpu().numpy()
    scale = 1 / np.sqrt(D)
    gots, refs = [], []
    for b, kv in [(0, 0), (3, 5), (7, 7)]:
        heads = slice(kv * G, (kv + 1) * G)
        refs.append(oatt.decode_rows(q[b, heads], ck[b, kv], cv[b, kv], oatt.head_params(params, kv), scale))
        gots.append(out[b, heads])
    assert_outputs_close(np.concatenate(gots), np.concatenate(refs), what="fp8 qwen3_8b full")


@pytest.mark.parametrize("shape", ["qwen3_8b", "gptoss_pair"])
def test_append_decode(nk, qwen8, gptoss8, shape):
    """The step call (one launch at head_dim 128): the new token's codes as the
    oracle's, the output as the oracle's, identical bits in both formats."""
    wl, params, P8, P16 = qwen8 if shape == "qwen3_8b" else gptoss8
    B, cap = 4, 2048
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    lens = np.array([1, 65, 1500, 2048], dtype=np.int32)
    ck = synth.random_codes(wl, 0, "k", (B, H, cap, L))
    cv = synth.random_codes(wl, 0, "v", (B, H, cap, L))
    kn = np.empty((B, H, D))
    vn = np.empty_like(kn)
    for b in range(B):
        for kv in range(H):
            kn[b, kv], vn[b, kv] = (x[0] for x in synth.cache_tokens(wl, 0, kv, b, 1, start=int(lens[b]) - 1))
    q = synth.decode_queries(wl, 0, batch=B)
    sinks = synth.sink_logits(wl, 0)
    res = []
    for P in (P8, P16):
        pk, pv = dev(ck, torch.uint8), dev(cv, torch.uint8)
        say(f"fp8 append+decode {shape} fp8={P.fp8_codebooks}")
        out = nk.append_decode_attn(P, nk.CacheLayout.contiguous(cap), dev(kn, torch.bfloat16),
                                    dev(vn, torch.bfloat16), dev(q, torch.bfloat16), pk, pv,
                                    dev(lens, torch.int32), cap,
                                    sinks=dev(sinks, torch.float32) if sinks is not None else None)
        torch.cuda.synchronize()
        res.append((out, pk, pv))
    assert torch.equal(res[0][0], res[1][0]) and torch.equal(res[0][1], res[1][1]) and torch.equal(res[0][2], res[1][2])
    out, pk, pv = (x.cpu().numpy() for x in res[0])
    scale = 1 / np.sqrt(D)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        p = int(lens[b]) - 1
        for kv in range(H):
            okk, ogk, ovv, ogv = ocodec.encode_tokens(kn[b, kv][None], vn[b, kv][None], oatt.head_params(params, kv))
            compare_codes(pk[b, kv, p:p + 1], okk, ogk, f"step b{b} kv{kv} K")
            compare_codes(pv[b, kv, p:p + 1], ovv, ogv, f"step b{b} kv{kv} V")
            rk, rv = ck[b, kv, :p + 1].copy(), cv[b, kv, :p + 1].copy()
            rk[p], rv[p] = okk[0], ovv[0]
            heads = slice(kv * G, (kv + 1) * G)
            ref[b, heads] = oatt.decode_rows(q[b, heads], rk, rv, oatt.head_params(params, kv), scale, 0,
                                             None if sinks is None else sinks[heads])
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D), what=f"fp8 step {shape}")


def test_key_scale_with_fp8_codebooks(nk):
    wl = synth.get_workload("qwen3_8b")
    params = calibrated_params(wl, 0, key_scale=True, fp8=True)
    P8, P16 = both_formats(nk, params, key_scale=True)
    B, n_new, cap = 2, 300, 512
    H, L, D, G = wl.num_kv_heads, wl.groups, wl.head_dim, wl.gqa
    kk = np.empty((B, n_new, H, D))
    vv = np.empty_like(kk)
    for b in range(B):
        for kv in range(H):
            kk[b, :, kv], vv[b, :, kv] = synth.cache_tokens(wl, 0, kv, b, n_new)
    lay = nk.CacheLayout.contiguous(cap)
    q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
    res = []
    for P in (P8, P16):
        pk = torch.zeros((B, H, cap, L), dtype=torch.uint8, device="cuda")
        pv = torch.zeros_like(pk)
        ps = torch.zeros((B, H, cap), dtype=torch.int16, device="cuda")
        say(f"fp8 key-scale encode+decode fp8={P.fp8_codebooks}")
        nk.encode(P, lay, dev(kk, torch.bfloat16), dev(vv, torch.bfloat16), dev([0, 0], torch.int32), pk, pv,
                  k_scales=ps)
        out = nk.decode_attn(P, lay, q, pk, pv, dev([n_new, n_new], torch.int32), cap, k_scales=ps)
        torch.cuda.synchronize()
        res.append((out, pk, pv, ps))
    for x, y in zip(res[0], res[1]):
        assert torch.equal(x, y)
    out, pk, pv, ps = res[0]
    hk, hs = pk.cpu().numpy(), ps.cpu().numpy().view(np.uint16)
    qh = synth.decode_queries(wl, 0, batch=B)
    ref = np.zeros(out.shape)
    for b in range(B):
        for kv in range(H):
            ck, gk, sb, cv, gv, rho = ocodec.encode_tokens_scaled(kk[b, :, kv], vv[b, :, kv],
                                                                  oatt.head_params(params, kv))
            compare_codes(hk[b, kv, :n_new], ck, gk, f"fp8 key-scale b{b} kv{kv} K")
            heads = slice(kv * G, (kv + 1) * G)
            ref[b, heads] = oatt.decode_rows(qh[b, heads], hk[b, kv, :n_new], pv.cpu().numpy()[b, kv, :n_new],
                                             oatt.head_params(params, kv), 1 / np.sqrt(D),
                                             scales_k=ocodec.bf16_value(hs[b, kv, :n_new]))
    assert_outputs_close(out.cpu().numpy().reshape(-1, D), ref.reshape(-1, D), what="fp8 key-scale decode")
