"""The one-launch step with a sink-plus-recent band, in every format.

With a band whose recent part holds the new token, nova_kv_append_decode_attn
runs as one launch of a table kernel (head_dim 128 or 64) in the plain, fp8,
key-scale and scalar-value formats and their combinations: encoder teams
store the new token's codes (and scale, levels, (scale, offset)), the split
that attends the band's last row stores that row, and the token is attended
exactly from it.

* against the two-call path (nova_kv_encode at seq_lens - 1, then
  nova_kv_decode_attn) on the same inputs: every written byte (codes, scales,
  scalar-arm words, band rows) identical, the outputs equal up to the
  rounding order of the dynamically claimed rounds;
* the deployed format (keys with a per-token scale, INT2 values, a 64 + 256
  band, sinks) against the oracle: the new token's codes, scale and levels,
  and the output (paper: Algorithm 1, write then attention; Sec. "Bit rate";
  Sec. "Sink-plus-recent band").
"""

import numpy as np
import pytest
import torch

import synth
from helpers import assert_outputs_close, compare_codes, row_errors
from oracle import attention as oatt
from oracle import codec as ocodec
from oracle import fp8 as ofp8
from oracle_cache import calibrated_params

pytestmark = pytest.mark.gpu

SAME_TOL = 5e-4  # fused vs two calls: only the rounding order of the splits' rounds differs


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


@pytest.fixture(scope="module")
def nk():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_04074_amd as nk
    nk._native.lib()
    return nk


def dev(x, dtype):
    return torch.as_tensor(np.ascontiguousarray(x)).to(dtype).cuda()


def dev_bits(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


FORMATS = {
    # name: (key scale, fp8 codebooks, scalar value arm)
    "band": (False, False, False),
    "band_fp8": (False, True, False),
    "key_scale": (True, False, False),
    "sq_values": (False, False, True),
    "deployed": (True, False, True),
    "deployed_fp8": (True, True, True),
}


def format_params(nk, wl, fmt):
    ks, f8, sq = FORMATS[fmt]
    params = calibrated_params(wl, 0, key_scale=ks, fp8=f8)
    arr = dict(params)
    if f8:
        arr["cb_k"] = ofp8.e4m3_bits(params["cb_k"].astype(np.float64))
        arr["cb_v"] = ofp8.e4m3_bits(params["cb_v"].astype(np.float64))
    if sq:
        arr["cb_v"] = None
    return params, nk.NovaKVParams.from_arrays(arr, key_scale=ks, sq_values=sq)


def history(wl, B, cap, n_sink, n_rec, seed):
    """Random codes, scales and scalar-arm words, and random finite band rows."""
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    rng = np.random.default_rng(seed)
    ck = synth.random_codes(wl, 0, "k", (B, H, cap, L))
    cv = rng.integers(0, 256, (B, H, cap, L), dtype=np.uint8)
    ks = synth.random_key_scales(wl, 0, (B, H, cap))
    sb = synth.random_key_scales(wl, 0, (B, H, cap), sigma=0.3)
    zb = ocodec.bf16_bits(-1.5 * ocodec.bf16_value(sb) + 0.2 * rng.standard_normal((B, H, cap)))
    band = ocodec.bf16_bits(rng.standard_normal((2, B, H, n_sink + n_rec, D)))
    return ck, cv, ks, np.stack([sb, zb], axis=-1), band


def run_both(nk, wl, P, fmt, lens, cap, *, window=0, sinks=None, n_sink=64, n_rec=256, seed=3, paged_bs=None,
             new_dtype=torch.bfloat16):
    """paged_bs: a paged cache of blocks of that many tokens (seeded shuffled
    block table; the history is then a random pool); new_dtype: the step's
    key and value (fp32 ones are rounded to bf16 for the band)."""
    ks, _, sq = FORMATS[fmt]
    B, H, D = len(lens), wl.num_kv_heads, wl.head_dim
    ck, cv, hks, hsq, hband = history(wl, B, cap, n_sink, n_rec, seed)
    rng = np.random.default_rng(seed + 1)
    kn = dev(rng.standard_normal((B, H, D)), new_dtype)
    vn = dev(rng.standard_normal((B, H, D)), new_dtype)
    q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
    lens_d = dev(np.asarray(lens, np.int32), torch.int32)
    sk = dev(sinks, torch.float32) if sinks is not None else None
    lay = nk.CacheLayout.contiguous(cap)
    if paged_bs:
        # the same bytes read as a pool of B * cap / paged_bs blocks of [Hkv][paged_bs] rows
        bps = cap // paged_bs
        table = np.random.default_rng(seed + 2).permutation(B * bps).astype(np.int32).reshape(B, bps)
        lay = nk.CacheLayout(paged_bs, bps, dev(table, torch.int32))
        ck = ck.reshape(B * bps, H, paged_bs, -1)
        cv = cv.reshape(B * bps, H, paged_bs, -1)
        hks = hks.reshape(B * bps, H, paged_bs)
        hsq = hsq.reshape(B * bps, H, paged_bs, 2)

    def state():
        return dict(k=dev(ck, torch.uint8), v=dev(cv, torch.uint8), ks=dev_bits(hks) if ks else None,
                    sq=dev_bits(hsq) if sq else None, bk=dev_bits(hband[0]), bv=dev_bits(hband[1]))

    one, two = state(), state()
    what = f"{fmt} B={B} cap={cap} window={window} band={n_sink}+{n_rec}" + (f" paged {paged_bs}" if paged_bs else "")
    say(f"deployed step {what}: one launch")
    out1 = nk.append_decode_attn(P, lay, kn, vn, q, one["k"], one["v"], lens_d, cap, window=window, sinks=sk,
                                 k_scales=one["ks"], v_sq=one["sq"], band=nk.Band(n_sink, n_rec, one["bk"], one["bv"]))
    say(f"deployed step {what}: encode, then decode")
    band2 = nk.Band(n_sink, n_rec, two["bk"], two["bv"])
    nk.encode(P, lay, kn[:, None], vn[:, None], lens_d - 1, two["k"], two["v"], k_scales=two["ks"], band=band2,
              v_sq=two["sq"])
    out2 = nk.decode_attn(P, lay, q, two["k"], two["v"], lens_d, cap, window=window, sinks=sk,
                          k_scales=two["ks"], v_sq=two["sq"], band=band2)
    torch.cuda.synchronize()
    for name in ("k", "v", "ks", "sq", "bk", "bv"):
        if one[name] is not None:
            assert torch.equal(one[name], two[name]), f"{fmt}: the one-launch step wrote other {name} bytes"
    o1, o2 = out1.cpu().numpy(), out2.cpu().numpy()
    assert np.isfinite(o1).all()
    err = row_errors(o1.reshape(-1, D), o2.reshape(-1, D).astype(np.float64))
    print(f"[parity] deployed step {what} vs two calls worst_rel_diff={float(err.max()):.3e}", flush=True)
    assert float(err.max()) <= SAME_TOL
    return one, o1


@pytest.mark.parametrize("fmt", list(FORMATS))
def test_step_matches_encode_then_decode(nk, fmt):
    wl = synth.get_workload("qwen3_8b")
    _, P = format_params(nk, wl, fmt)
    sinks = np.random.default_rng(4).standard_normal(wl.num_q_heads).astype(np.float32)
    # ragged lengths: a one-token sequence (only the new token, a sink slot),
    # one inside the sinks, one just past the band, long ones
    run_both(nk, wl, P, fmt, [1, 40, 330, 2048], 2048, sinks=sinks)
    run_both(nk, wl, P, fmt, [1500, 2048, 700, 321], 2048, window=500, seed=5)


@pytest.mark.parametrize("fmt", ["band", "deployed", "deployed_fp8"])
def test_step_paged_fp32_inputs(nk, fmt):
    """A paged cache of 16-token blocks (shuffled table) and fp32 step inputs."""
    wl = synth.get_workload("qwen3_8b")
    _, P = format_params(nk, wl, fmt)
    run_both(nk, wl, P, fmt, [1, 333, 2048, 1000], 2048, window=700, paged_bs=16, new_dtype=torch.float32, seed=8)


@pytest.mark.parametrize("paged_bs", [None, 16], ids=["contiguous", "paged16"])
@pytest.mark.parametrize("fmt", ["band", "deployed"])
def test_step_one_split_per_unit(nk, fmt, paged_bs):
    """32 sequences x 8 KV heads fill the 256 workgroups with one split per
    (sequence, KV head): the contiguous step stays one launch, the paged one
    runs as encode then decode; both store the encoder's bytes and give the
    decode's output."""
    wl = synth.get_workload("qwen3_8b")
    _, P = format_params(nk, wl, fmt)
    lens = [1024, 1, 333, 1023, 700, 64, 512, 999] * 4
    run_both(nk, wl, P, fmt, lens, 1024, paged_bs=paged_bs, seed=11)


@pytest.mark.parametrize("fmt", ["band", "deployed"])
def test_step_with_sinks_only(nk, fmt):
    """A band of sink positions only (n_rec = 0): the new token is read from
    codes, so the step runs as the encode and then the decode."""
    wl = synth.get_workload("qwen3_8b")
    _, P = format_params(nk, wl, fmt)
    run_both(nk, wl, P, fmt, [1, 40, 64, 65, 2048], 2048, n_sink=64, n_rec=0, seed=9)


@pytest.mark.parametrize("fmt", ["band", "key_scale", "sq_values", "deployed", "deployed_fp8"])
def test_head_dim_64_step(nk, fmt):
    """The GPT-OSS shape (head_dim 64, eight query heads per KV head, learned
    sinks) on its table kernel: the first split to count in encodes the new
    token, the combining split stores and attends its band row.  Ragged
    lengths, a window of 128, many splits per KV head."""
    wl = synth.get_workload("gptoss_pair")
    _, P = format_params(nk, wl, fmt)
    sinks = synth.sink_logits(wl, 0)
    run_both(nk, wl, P, fmt, [1, 40, 330, 2048], 2048, sinks=sinks)
    run_both(nk, wl, P, fmt, [2048, 1500, 700, 321], 2048, window=128, sinks=sinks, seed=5)
    run_both(nk, wl, P, fmt, [32768, 30000], 32768, sinks=sinks, seed=6)


@pytest.mark.parametrize("fmt", ["band", "deployed"])
@pytest.mark.parametrize("B,S", [(8, 16384), (1, 16384)], ids=["bench_shape", "one_sequence"])
def test_step_matches_at_many_splits(nk, fmt, B, S):
    """The bench shape (4 splits per KV head, the tasks spread over them) and
    one sequence (32 splits in groups, the band shared by many splits)."""
    wl = synth.get_workload("qwen3_8b")
    _, P = format_params(nk, wl, fmt)
    sinks = np.random.default_rng(4).standard_normal(wl.num_q_heads).astype(np.float32)
    run_both(nk, wl, P, fmt, [S - 7 * i for i in range(B)], S, sinks=sinks)


@pytest.mark.parametrize("shape", ["qwen3_8b", "gptoss_pair"])
def test_deployed_step_against_the_oracle(nk, shape):
    wl = synth.get_workload(shape)
    params, P = format_params(nk, wl, "deployed")
    n_sink, n_rec = 64, 256
    B, cap = 4, 2304
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    lens = np.array([1, 65, 1500, 2304], dtype=np.int32)
    ck, cv, hks, hsq, _ = history(wl, B, cap, n_sink, n_rec, 11)
    band_k = np.full((B, H, n_sink + n_rec, D), 0x7FC0, dtype=np.uint16)  # NaN where nothing is attended
    band_v = band_k.copy()
    exact = {}
    for b in range(B):
        S = int(lens[b])
        for kv in range(H):
            kx, vx = synth.cache_tokens(wl, 0, kv, b, S)
            exact[b, kv] = (ocodec.band_values(kx), ocodec.band_values(vx))
            for p in np.flatnonzero(oatt.band_mask(S - 1, n_sink, n_rec)):  # the band before the step's token
                sl = p if p < n_sink else n_sink + p % n_rec
                band_k[b, kv, sl] = ocodec.bf16_bits(kx[p])
                band_v[b, kv, sl] = ocodec.bf16_bits(vx[p])
    kn = np.stack([[exact[b, kv][0][int(lens[b]) - 1] for kv in range(H)] for b in range(B)])
    vn = np.stack([[exact[b, kv][1][int(lens[b]) - 1] for kv in range(H)] for b in range(B)])
    q = synth.decode_queries(wl, 0, batch=B)
    sinks = np.random.default_rng(4).standard_normal(wl.num_q_heads).astype(np.float32)  # learned-sink logits
    pk, pv, pks, psq = dev(ck, torch.uint8), dev(cv, torch.uint8), dev_bits(hks), dev_bits(hsq)
    bk, bv = dev_bits(band_k), dev_bits(band_v)
    say(f"deployed step against the oracle {shape}")
    out = nk.append_decode_attn(P, nk.CacheLayout.contiguous(cap), dev(kn, torch.bfloat16), dev(vn, torch.bfloat16),
                                dev(q, torch.bfloat16), pk, pv, dev(lens, torch.int32), cap,
                                sinks=dev(sinks, torch.float32), k_scales=pks, v_sq=psq,
                                band=nk.Band(n_sink, n_rec, bk, bv)).cpu().numpy()
    assert np.isfinite(out).all()
    hk, hv = pk.cpu().numpy(), pv.cpu().numpy()
    hs = pks.cpu().numpy().view(np.uint16)
    hq = psq.cpu().numpy().view(np.uint16)
    hbk, hbv = bk.cpu().numpy().view(np.uint16), bv.cpu().numpy().view(np.uint16)
    scale = 1 / np.sqrt(D)
    ref = np.zeros_like(out, dtype=np.float64)
    from test_gpu_sq import compare_sq, near_bits
    for b in range(B):
        S = int(lens[b])
        p = S - 1
        for kv in range(H):
            hp = oatt.head_params(params, kv)
            kb, vb = exact[b, kv]
            sl = p if p < n_sink else n_sink + p % n_rec
            assert np.array_equal(hbk[b, kv, sl], ocodec.bf16_bits(kb[p])), f"b{b} kv{kv}: band key row"
            assert np.array_equal(hbv[b, kv, sl], ocodec.bf16_bits(vb[p])), f"b{b} kv{kv}: band value row"
            okk, ogk, _, _, _, rho = ocodec.encode_tokens_scaled(kb[p][None], vb[p][None], hp)
            compare_codes(hk[b, kv, p:p + 1], okk, ogk, f"deployed step {shape} b{b} kv{kv} K")
            assert near_bits(hs[b, kv, p:p + 1], rho).all(), f"b{b} kv{kv}: key scale"
            compare_sq(hv[b, kv, p:p + 1], hq[b, kv, p:p + 1, 0], hq[b, kv, p:p + 1, 1], vb[p][None], hp["t_v"],
                       f"deployed step {shape} b{b} kv{kv} V")
            heads = slice(kv * G, (kv + 1) * G)
            ref[b, heads] = oatt.decode_rows(q[b, heads], hk[b, kv, :S], hv[b, kv, :S], hp, scale, 0, sinks[heads],
                                             scales_k=ocodec.bf16_value(hs[b, kv, :S]),
                                             band=(n_sink, n_rec, kb[:S], vb[:S]),
                                             sq_v=(hq[b, kv, :S, 0], hq[b, kv, :S, 1]))
    assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D), what=f"deployed step {shape}")
