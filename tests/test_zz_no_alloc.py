"""The allocation-free step (nova_kv_append_decode_attn_noalloc) against the
step with a caller's workspace, on two calls in a row, the second with a
smaller input: the stored codes bit-exact, the outputs within the parity
tolerance (splits of more than twelve rounds hand their later rounds to
whichever wave is free, so two runs of the same step agree up to rounding)."""

import numpy as np
import pytest
import torch

import synth
from helpers import assert_outputs_close
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


def _step_both(nk, wl, P, B, cap, lens, seed):
    H, L, D, Hq = wl.num_kv_heads, wl.groups, wl.head_dim, wl.num_q_heads
    ck = synth.random_codes(wl, 0, "k", (B, H, cap, L))
    cv = synth.random_codes(wl, 0, "v", (B, H, cap, L))
    rng = np.random.default_rng(seed)
    kn, vn = rng.standard_normal((2, B, H, D))
    q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
    sinks = dev(synth.sink_logits(wl, 0), torch.float32) if wl.sinks else None
    lay = nk.CacheLayout.contiguous(cap)
    lens_d = dev(lens, torch.int32)
    kn_d, vn_d = dev(kn, torch.bfloat16), dev(vn, torch.bfloat16)
    window = wl.windows[0]
    say(f"{wl.name} B={B} cap={cap}: step with a workspace")
    pk1, pv1 = dev(ck, torch.uint8), dev(cv, torch.uint8)
    out1 = nk.append_decode_attn(P, lay, kn_d, vn_d, q, pk1, pv1, lens_d, cap, window=window, sinks=sinks)
    say(f"{wl.name} B={B} cap={cap}: allocation-free step")
    pk2, pv2 = dev(ck, torch.uint8), dev(cv, torch.uint8)
    out2 = torch.empty_like(out1)
    nk.append_decode_attn_noalloc(P, lay, kn_d, vn_d, q, pk2, pv2, lens_d, cap, out2, window=window, sinks=sinks)
    torch.cuda.synchronize()
    assert torch.equal(pk1, pk2) and torch.equal(pv1, pv2)
    assert torch.isfinite(out2).all()
    assert_outputs_close(out2.cpu().numpy().reshape(-1, D), out1.cpu().numpy().reshape(-1, D).astype(np.float64),
                         what=f"noalloc vs workspace {wl.name} B={B} cap={cap}")
    return float((out2 - out1).abs().max())


@pytest.mark.parametrize("shape", ["qwen3_8b", "gptoss_pair"])
def test_noalloc_step_matches_the_workspace_step(nk, shape):
    wl = synth.get_workload(shape)
    P = nk.NovaKVParams.from_arrays(calibrated_params(wl, 0))
    # two calls in a row on the shared scratch, the second smaller
    d1 = _step_both(nk, wl, P, 4, 8192, np.array([8192, 5001, 64, 1], dtype=np.int32), 1)
    d2 = _step_both(nk, wl, P, 2, 2048, np.array([2048, 700], dtype=np.int32), 2)
    print(f"[parity] noalloc {shape} max_abs_diff first={d1:.3e} second={d2:.3e}", flush=True)


def test_noalloc_step_rejects_shapes_beyond_its_scratch(nk):
    wl = synth.get_workload("qwen3_8b")
    P = nk.NovaKVParams.from_arrays(calibrated_params(wl, 0))
    B, cap = 64, 32768
    assert nk.decode_workspace_bytes(P, B, wl.num_q_heads, cap) > nk.NOALLOC_SCRATCH_BYTES
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    pk = torch.zeros((1, H, 16, L), dtype=torch.uint8, device="cuda")
    lay = nk.CacheLayout(16, cap // 16, torch.zeros((B, cap // 16), dtype=torch.int32, device="cuda"))
    x = torch.zeros((B, H, D), dtype=torch.bfloat16, device="cuda")
    q = torch.zeros((B, wl.num_q_heads, D), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((B, wl.num_q_heads, D), dtype=torch.float32, device="cuda")
    lens = torch.ones(B, dtype=torch.int32, device="cuda")
    with pytest.raises(nk.NovaKVError, match="allocation-free"):
        nk.append_decode_attn_noalloc(P, lay, x, x, q, pk, pk, lens, cap, out)
