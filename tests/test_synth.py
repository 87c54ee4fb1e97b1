"""The seeded input generator: determinism, storage rounding, spectra, block tables."""

import numpy as np
import torch

import synth


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 37
    ours = synth.round_to_bf16(x)
    ref = torch.tensor(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours, ref)


def test_spectrum_and_bases():
    lam = synth.power_spectrum(128, 1.0)
    assert np.isclose(lam.sum(), 128) and np.all(np.diff(lam) < 0)
    assert np.isclose(lam[0] / lam[1], 2.0)
    wl = synth.get_workload("gptoss_pair")
    u_k, u_v, u_q = synth.head_bases(wl, 1, 3)
    for u in (u_k, u_v, u_q):
        assert np.allclose(u @ u.T, np.eye(64), atol=1e-12)
    assert not np.allclose(u_q, u_k)
    wl2 = synth.get_workload("qwen3_8b")
    a, _, c = synth.head_bases(wl2, 0, 0)
    assert np.array_equal(a, c)


def test_deterministic_and_subrange_consistent():
    wl = synth.get_workload("qwen3_8b")
    k1, v1 = synth.cache_tokens(wl, 0, 2, 3, 3000)
    k2, v2 = synth.cache_tokens(wl, 0, 2, 3, 1000, start=1500)
    assert np.array_equal(k1[1500:2500], k2) and np.array_equal(v1[1500:2500], v2)
    assert np.array_equal(synth.round_to_bf16(k1).astype(np.float64), k1)


def test_block_table_is_a_permutation():
    wl = synth.get_workload("append_paged")
    bt = synth.shuffled_block_table(wl)
    assert bt.shape == (32, 2048)
    assert np.array_equal(np.sort(bt.ravel()), np.arange(32 * 2048))


def test_device_cache_tokens_are_seeded_and_follow_the_model():
    """The device-side generator (run here on the CPU device) is reproducible,
    depends on the sequence and start, and draws each KV head's tokens with
    that head's basis and spectrum."""
    wl = synth.get_workload("append_paged")
    k, v = synth.device_cache_tokens(wl, 0, 3, 8192, 1024, "cpu")
    k2, v2 = synth.device_cache_tokens(wl, 0, 3, 8192, 1024, "cpu")
    assert k.dtype == torch.bfloat16 and tuple(k.shape) == (8192, 8, 128)
    assert torch.equal(k, k2) and torch.equal(v, v2)
    assert not torch.equal(k, synth.device_cache_tokens(wl, 0, 4, 8192, 1024, "cpu")[0])
    lam = synth.power_spectrum(128, 1.0)
    for kv in (0, 5):
        u_k, u_v, _ = synth.head_bases(wl, 0, kv)
        for x, u in ((k[:, kv], u_k), (v[:, kv], u_v)):
            var = (x.double().numpy() @ u).var(axis=0)
            # 8192 draws: relative standard error of a variance ~ sqrt(2 / 8192) = 1.6%
            assert np.all(np.abs(var / lam - 1) < 0.08)
