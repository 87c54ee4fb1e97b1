"""Decode calls captured in a HIP graph and replayed.

A replay repeats the captured call's arguments, the split exchange's tag
(epoch) included.  In a captured call the head_dim-128 table kernel's
combining workgroups empty every exchange word they read, so each replay
leaves its part of the workspace all zero (the arrival counters are reset by
their last arrival) and never meets a word of the replay before; directly
launched calls leave their words, under odd epochs that no captured call
uses.  Every replay here gets new inputs in the captured buffers, shares its
workspace with a direct call on the same inputs made right after it, must
match that call (up to the rounding of the dynamically claimed rounds), and
must leave the workspace all zero.  Cases: one-level combine, two-level
combine with a sink-plus-recent band, the fused one-launch step (with a
workspace and allocation-free), and the head_dim-64 table kernel (whose
splits complete their stores before counting in)."""

import numpy as np
import pytest
import torch

import synth
from helpers import row_errors
from oracle_cache import calibrated_params

pytestmark = pytest.mark.gpu

REPLAYS = 3
TOL = 1e-3  # row max-abs difference relative to the row norm; a stale word errs by O(1)


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


def close(got, ref, what):
    D = got.shape[-1]
    g = got.cpu().numpy()
    assert np.isfinite(g).all(), what
    err = row_errors(g.reshape(-1, D), ref.cpu().numpy().reshape(-1, D).astype(np.float64))
    worst = float(err.max()) if err.size else 0.0
    print(f"[graph] {what} worst_rel_diff={worst:.3e}", flush=True)
    assert worst <= TOL, f"{what}: replay differs from the direct call ({worst:.3e})"


def shape(nk, name, **scaled):
    wl = synth.get_workload(name)
    params = calibrated_params(wl, 0)
    if scaled:
        wl = wl.scaled(**scaled)
        params = {k: v[: wl.num_kv_heads] for k, v in params.items()}
    return wl, nk.NovaKVParams.from_arrays(params)


def pools(wl, B, cap):
    H, L = wl.num_kv_heads, wl.groups
    return (dev(synth.random_codes(wl, 0, "k", (B, H, cap, L)), torch.uint8),
            dev(synth.random_codes(wl, 0, "v", (B, H, cap, L)), torch.uint8))


def band_of(nk, wl, B, n_sink, n_rec, seed):
    rng = np.random.default_rng(seed)
    shp = (B, wl.num_kv_heads, n_sink + n_rec, wl.head_dim)
    k = torch.as_tensor(rng.standard_normal(shp), dtype=torch.bfloat16).cuda()
    v = torch.as_tensor(rng.standard_normal(shp), dtype=torch.bfloat16).cuda()
    return nk.Band(n_sink, n_rec, k, v)


def new_inputs(wl, B, r):
    rng = np.random.default_rng(100 + r)
    q = rng.standard_normal((B, wl.num_q_heads, wl.head_dim))
    kn, vn = rng.standard_normal((2, B, wl.num_kv_heads, wl.head_dim))
    return dev(q, torch.bfloat16), dev(kn, torch.bfloat16), dev(vn, torch.bfloat16)


def workspace_zero(ws, what):
    torch.cuda.synchronize()
    assert int(ws.count_nonzero()) == 0, f"{what}: exchange words left behind"


def run_decode_case(nk, wl, P, B, cap, lens, what, band=None):
    kp, vp = pools(wl, B, cap)
    lay = nk.CacheLayout.contiguous(cap)
    lens_d = dev(lens, torch.int32)
    ws = torch.zeros(nk.decode_workspace_bytes(P, B, wl.num_q_heads, cap), dtype=torch.uint8, device="cuda")
    q_g = torch.zeros((B, wl.num_q_heads, wl.head_dim), dtype=torch.bfloat16, device="cuda")
    out_g = torch.zeros((B, wl.num_q_heads, wl.head_dim), dtype=torch.float32, device="cuda")
    say(f"graph decode {what}: direct call, then capture")
    nk.decode_attn(P, lay, new_inputs(wl, B, 0)[0], kp, vp, lens_d, cap, workspace=ws, band=band)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        nk.decode_attn(P, lay, q_g, kp, vp, lens_d, cap, out=out_g, workspace=ws, band=band)
    torch.cuda.synchronize()
    for r in range(REPLAYS):
        q, _, _ = new_inputs(wl, B, r + 1)
        q_g.copy_(q)
        say(f"graph decode {what}: replay {r}")
        g.replay()
        if wl.head_dim == 128:
            workspace_zero(ws, f"{what} replay {r}")
        ref = nk.decode_attn(P, lay, q, kp, vp, lens_d, cap, workspace=ws, band=band)
        torch.cuda.synchronize()
        close(out_g, ref, f"{what} replay {r}")


def test_one_level_replays(nk):
    wl, P = shape(nk, "qwen3_8b")
    run_decode_case(nk, wl, P, 8, 8192, np.array([8192, 8000, 5000, 4097, 2048, 700, 64, 1], np.int32),
                    "qwen3_8b B=8 (4 splits)")


def test_two_level_band_replays(nk):
    wl, P = shape(nk, "qwen3_8b", num_kv_heads=2, num_q_heads=8)
    run_decode_case(nk, wl, P, 2, 65536, np.array([65536, 40000], np.int32),
                    "two KV heads B=2 S=65536 (64 splits, band)", band=band_of(nk, wl, 2, 64, 256, 7))


def test_head_dim_64_replays(nk):
    wl, P = shape(nk, "gptoss_pair")
    run_decode_case(nk, wl, P, 4, 8192, np.array([8192, 5000, 700, 1], np.int32), "gptoss B=4")


@pytest.mark.parametrize("noalloc", [False, True], ids=["workspace", "noalloc"])
@pytest.mark.parametrize("B,cap", [(4, 8192), (1, 32768)], ids=["one_level", "two_level"])
def test_fused_step_replays(nk, noalloc, B, cap):
    wl, P = shape(nk, "qwen3_8b")
    what = f"fused step B={B} cap={cap} {'noalloc' if noalloc else 'workspace'}"
    kp_g, vp_g = pools(wl, B, cap)
    kp_e, vp_e = kp_g.clone(), vp_g.clone()
    lay = nk.CacheLayout.contiguous(cap)
    lens_d = dev(np.array([cap, cap - 300, 4097, 1][:B], np.int32), torch.int32)
    ws = torch.zeros(nk.decode_workspace_bytes(P, B, wl.num_q_heads, cap), dtype=torch.uint8, device="cuda")
    shp_q, shp_kv = (B, wl.num_q_heads, wl.head_dim), (B, wl.num_kv_heads, wl.head_dim)
    q_g = torch.zeros(shp_q, dtype=torch.bfloat16, device="cuda")
    kn_g = torch.zeros(shp_kv, dtype=torch.bfloat16, device="cuda")
    vn_g = torch.zeros(shp_kv, dtype=torch.bfloat16, device="cuda")
    out_g = torch.zeros(shp_q, dtype=torch.float32, device="cuda")

    def direct(q, kn, vn, kp, vp, out=None):
        # the direct calls share the captured call's scratch (its workspace, or the GPU's array)
        if noalloc:
            out = torch.empty_like(out_g) if out is None else out
            nk.append_decode_attn_noalloc(P, lay, kn, vn, q, kp, vp, lens_d, cap, out)
            return out
        return nk.append_decode_attn(P, lay, kn, vn, q, kp, vp, lens_d, cap, out=out, workspace=ws)

    # a direct step first (also the allocation-free step's first call on the
    # device, which looks its array up and clears it outside the capture)
    say(f"graph {what}: direct step, then capture")
    q0, kn0, vn0 = new_inputs(wl, B, 0)
    direct(q0, kn0, vn0, kp_g, vp_g)
    direct(q0, kn0, vn0, kp_e, vp_e)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        direct(q_g, kn_g, vn_g, kp_g, vp_g, out=out_g)
    torch.cuda.synchronize()
    for r in range(REPLAYS):
        q, kn, vn = new_inputs(wl, B, r + 1)
        q_g.copy_(q)
        kn_g.copy_(kn)
        vn_g.copy_(vn)
        say(f"graph {what}: replay {r}")
        g.replay()
        if not noalloc:
            workspace_zero(ws, f"{what} replay {r}")
        ref = direct(q, kn, vn, kp_e, vp_e)
        torch.cuda.synchronize()
        assert torch.equal(kp_g, kp_e) and torch.equal(vp_g, vp_e), f"{what}: replay {r} stored other codes"
        close(out_g, ref, f"{what} replay {r}")
