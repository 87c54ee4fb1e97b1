"""Transforms stored as bf16 (NOVA_KV_BF16_TRANSFORMS; paper: Sec.
"Calibration", the bases are cast to bfloat16 when loaded into the serving
engine).  Every kernel reads t_k, t_k_inv_t and t_v as those exact bf16
values, so the oracle, given the same rounded matrices, is the reference:
codes bit-exact up to near-ties, outputs within 2e-3 of the row norm, on the
head_dim-128 and head_dim-64 table kernels, the split-K kernels, both
encoders, the scalar-arm encoder and both one-launch steps."""

import numpy as np
import pytest
import torch

import synth
from helpers import assert_outputs_close, compare_codes, read_rows, row_errors
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
    nk._native.lib()
    return nk


def dev(x, dtype):
    return torch.as_tensor(np.ascontiguousarray(x)).to(dtype).cuda()


def bf16_round(x):
    """fp64 copy of x rounded to bf16 (nearest even, through fp32, as the binding stores it)."""
    return torch.as_tensor(np.asarray(x, dtype=np.float64)).to(torch.float32).to(torch.bfloat16) \
        .to(torch.float64).numpy()


def rounded_params(wl, **kw):
    params = calibrated_params(wl, 0, **kw)
    return dict(params, **{k: bf16_round(params[k]) for k in ("t_k", "t_k_inv_t", "t_v")})


def test_the_binding_stores_bf16(nk):
    wl = synth.get_workload("qwen3_8b")
    params = rounded_params(wl)
    P = nk.NovaKVParams.from_arrays(params, bf16_transforms=True)
    assert P.bf16_transforms and P.t_k.dtype == torch.bfloat16 and P.kbar.dtype == torch.float32
    assert P.c.flags & nk._native.NOVA_KV_BF16_TRANSFORMS
    # the rounded values are stored exactly
    assert np.array_equal(P.t_k_inv_t.cpu().to(torch.float64).numpy(), params["t_k_inv_t"])


@pytest.mark.parametrize("shape", ["qwen3_8b", "gptoss_pair"])
@pytest.mark.parametrize("block_size", [None, 8], ids=["table", "split_k"])
def test_encode_then_decode(nk, shape, block_size):
    """Encode (bulk, then one token) into the pools, decode ragged lengths with
    a window and sinks; block_size 8 takes the split-K decode."""
    wl = synth.get_workload(shape)
    params = rounded_params(wl)
    P = nk.NovaKVParams.from_arrays(params, bf16_transforms=True)
    B, cap, n0 = 3, 1024, 999
    H, L, G, D = wl.num_kv_heads, wl.groups, wl.gqa, wl.head_dim
    kk = np.empty((B, cap, H, D))
    vv = np.empty_like(kk)
    for b in range(B):
        for kv in range(H):
            kk[b, :, kv], vv[b, :, kv] = synth.cache_tokens(wl, 0, kv, b, cap)
    if block_size:
        bps = cap // block_size
        table = np.random.default_rng(5).permutation(B * bps).astype(np.int32).reshape(B, bps)
        lay = nk.CacheLayout(block_size, bps, dev(table, torch.int32))
        lk = dict(hkv=H, block_size=block_size, blocks_per_seq=bps, table=table)
        pk = torch.zeros((B * bps, H, block_size, L), dtype=torch.uint8, device="cuda")
    else:
        lay = nk.CacheLayout.contiguous(cap)
        lk = dict(hkv=H, block_size=cap, blocks_per_seq=1, table=None)
        pk = torch.zeros((B, H, cap, L), dtype=torch.uint8, device="cuda")
    pv = torch.zeros_like(pk)
    say(f"bf16 transforms {shape} block_size={block_size}: encode")
    nk.encode(P, lay, dev(kk[:, :n0], torch.bfloat16), dev(vv[:, :n0], torch.bfloat16), dev([0] * B, torch.int32),
              pk, pv)
    nk.encode(P, lay, dev(kk[:, n0:], torch.bfloat16), dev(vv[:, n0:], torch.bfloat16), dev([n0] * B, torch.int32),
              pk, pv)
    torch.cuda.synchronize()
    hk, hv = pk.cpu().numpy().reshape(-1), pv.cpu().numpy().reshape(-1)
    codes = {}
    for b in range(B):
        for kv in range(H):
            hp = oatt.head_params(params, kv)
            ck, gk, cv, gv = ocodec.encode_tokens(kk[b, :, kv], vv[b, :, kv], hp)
            compare_codes(read_rows(hk, b, kv, 0, cap, groups=L, **lk), ck, gk, f"bf16 T {shape} b{b} kv{kv} K")
            compare_codes(read_rows(hv, b, kv, 0, cap, groups=L, **lk), cv, gv, f"bf16 T {shape} b{b} kv{kv} V")
            codes[b, kv] = (read_rows(hk, b, kv, 0, cap, groups=L, **lk), read_rows(hv, b, kv, 0, cap, groups=L, **lk))
    lens = np.array([1, 700, 1024], dtype=np.int32)
    q = synth.decode_queries(wl, 0, batch=B)
    sinks = np.random.default_rng(2).standard_normal(wl.num_q_heads).astype(np.float32)
    scale = 1 / np.sqrt(D)
    for window in (0, 300):
        say(f"bf16 transforms {shape} block_size={block_size}: decode window={window}")
        out = nk.decode_attn(P, lay, dev(q, torch.bfloat16), pk, pv, dev(lens, torch.int32), cap, window=window,
                             sinks=dev(sinks, torch.float32)).cpu().numpy()
        ref = np.zeros_like(out, dtype=np.float64)
        for b in range(B):
            S = int(lens[b])
            for kv in range(H):
                heads = slice(kv * G, (kv + 1) * G)
                ck, cv = codes[b, kv]
                ref[b, heads] = oatt.decode_rows(q[b, heads], ck[:S], cv[:S], oatt.head_params(params, kv), scale,
                                                 window, sinks[heads])
        assert_outputs_close(out.reshape(-1, D), ref.reshape(-1, D),
                             what=f"bf16 transforms {shape} block_size={block_size} window={window}")


@pytest.mark.parametrize("shape,fmt", [("qwen3_8b", "plain"), ("qwen3_8b", "deployed"), ("gptoss_pair", "deployed")])
def test_step_matches_encode_then_decode(nk, shape, fmt):
    """The one-launch step (plain; the deployed format with a band) against the
    encode then the decode, every written byte equal."""
    wl = synth.get_workload(shape)
    deployed = fmt == "deployed"
    params = rounded_params(wl, key_scale=deployed)
    arr = dict(params, cb_v=None) if deployed else params
    P = nk.NovaKVParams.from_arrays(arr, key_scale=deployed, sq_values=deployed, bf16_transforms=True)
    B, cap = 4, 2048
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    rng = np.random.default_rng(12)
    ck = synth.random_codes(wl, 0, "k", (B, H, cap, L))
    cv = rng.integers(0, 256, (B, H, cap, L), dtype=np.uint8)
    ks = synth.random_key_scales(wl, 0, (B, H, cap))
    sq = np.stack([synth.random_key_scales(wl, 0, (B, H, cap), sigma=0.3),
                   ocodec.bf16_bits(0.2 * rng.standard_normal((B, H, cap)))], axis=-1)
    band = ocodec.bf16_bits(rng.standard_normal((2, B, H, 64 + 256, D)))
    kn = dev(rng.standard_normal((B, H, D)), torch.bfloat16)
    vn = dev(rng.standard_normal((B, H, D)), torch.bfloat16)
    q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
    lens = dev(np.array([1, 333, 1500, 2048], np.int32), torch.int32)
    lay = nk.CacheLayout.contiguous(cap)
    bits = lambda x: torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).cuda()  # noqa: E731

    def state():
        st = dict(k=dev(ck, torch.uint8), v=dev(cv, torch.uint8))
        if deployed:
            st.update(ks=bits(ks), sq=bits(sq), bk=bits(band[0]), bv=bits(band[1]))
        return st

    one, two = state(), state()
    kw1 = dict(k_scales=one["ks"], v_sq=one["sq"], band=nk.Band(64, 256, one["bk"], one["bv"])) if deployed else {}
    kw2 = dict(k_scales=two["ks"], v_sq=two["sq"], band=nk.Band(64, 256, two["bk"], two["bv"])) if deployed else {}
    say(f"bf16 transforms step {shape} {fmt}")
    out1 = nk.append_decode_attn(P, lay, kn, vn, q, one["k"], one["v"], lens, cap, **kw1)
    nk.encode(P, lay, kn[:, None], vn[:, None], lens - 1, two["k"], two["v"], k_scales=kw2.get("k_scales"),
              band=kw2.get("band"), v_sq=kw2.get("v_sq"))
    out2 = nk.decode_attn(P, lay, q, two["k"], two["v"], lens, cap, **kw2)
    torch.cuda.synchronize()
    for name in one:
        assert torch.equal(one[name], two[name]), f"{shape} {fmt}: the step wrote other {name} bytes"
    err = row_errors(out1.cpu().numpy().reshape(-1, D), out2.cpu().numpy().reshape(-1, D).astype(np.float64))
    print(f"[parity] bf16 transforms step {shape} {fmt} vs two calls worst_rel_diff={float(err.max()):.3e}",
          flush=True)
    assert float(err.max()) <= 5e-4
