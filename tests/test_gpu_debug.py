"""Debug mode of the entry points: the metadata is copied to the host and
checked before a launch.  Each rejected input below would also be harmless
if it were launched (its reads and writes stay inside the allocated pools),
so the test does not depend on the check to keep the GPU safe."""

import numpy as np
import pytest
import torch

import synth
from oracle_cache import calibrated_params

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


@pytest.fixture(scope="module")
def nk():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2608_04074_amd as nk
    nk._native.lib()
    yield nk
    nk.set_debug(False)


def dev(x, dtype):
    return torch.as_tensor(np.ascontiguousarray(x)).to(dtype).cuda()


def test_debug_mode_checks_metadata_before_launching(nk):
    wl = synth.get_workload("qwen3_8b")
    P = nk.NovaKVParams.from_arrays(calibrated_params(wl, 0))
    B, bs, bps = 2, 16, 160          # capacity 2560 per sequence; the pools hold 8 spare blocks
    H, L, D = wl.num_kv_heads, wl.groups, wl.head_dim
    nblocks = B * bps + 8
    table = np.random.default_rng(3).permutation(nblocks)[: B * bps].astype(np.int32).reshape(B, bps)
    rng = np.random.default_rng(4)
    pk = dev(rng.integers(0, 256, (nblocks, H, bs, L)), torch.uint8)
    pv = dev(rng.integers(0, 256, (nblocks, H, bs, L)), torch.uint8)
    q = dev(synth.decode_queries(wl, 0, batch=B), torch.bfloat16)
    lay = nk.CacheLayout(bs, bps, dev(table, torch.int32))
    good = dev([2048, 700], torch.int32)
    try:
        say("debug off: reference decode")
        ref = nk.decode_attn(P, lay, q, pk, pv, good, 2048)
        nk.set_debug(True, nblocks)
        say("debug on: valid decode")
        out = nk.decode_attn(P, lay, q, pk, pv, good, 2048)
        assert torch.equal(out, ref)
        say("debug on: a length past max_seq_len")
        with pytest.raises(nk.NovaKVError, match="debug mode: seq_lens\\[1\\] = 2049"):
            nk.decode_attn(P, lay, q, pk, pv, dev([2048, 2049], torch.int32), 2048)
        say("debug on: a block-table entry past the declared pool")
        nk.set_debug(True, B * bps)
        bad = table.copy()
        bad[0, 3] = B * bps + 2          # allocated, but beyond the declared pool size
        with pytest.raises(nk.NovaKVError, match="physical block"):
            nk.decode_attn(P, nk.CacheLayout(bs, bps, dev(bad, torch.int32)), q, pk, pv, good, 2048)
        say("debug on: an encode past the capacity")
        kk = dev(rng.standard_normal((B, 4, H, D)), torch.bfloat16)
        before = pk.clone()
        with pytest.raises(nk.NovaKVError, match="writes positions \\[2558, 2562\\)"):
            nk.encode(P, lay, kk, kk, dev([0, bs * bps - 2], torch.int32), pk, pv)
        torch.cuda.synchronize()
        assert torch.equal(pk, before)   # nothing was launched
        say("debug on: two sequences appending into one row")
        shared = table.copy()
        shared[1, 0] = shared[0, 0]
        kn = kk[:, 0].contiguous()
        with pytest.raises(nk.NovaKVError, match="write the same row"):
            nk.append_decode_attn(P, nk.CacheLayout(bs, bps, dev(shared, torch.int32)), kn, kn, q,
                                  pk, pv, dev([1, 1], torch.int32), 2048)
    finally:
        nk.set_debug(False)
