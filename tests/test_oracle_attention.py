"""Pins for the oracle's decode attention (plain form), against a library SDPA."""

import numpy as np
import pytest
import torch

from oracle import attention as att
from oracle import codec, vq


def _sdpa(q, k, v, scale):
    """Library reference: torch scaled_dot_product_attention in fp64 on the CPU."""
    qt = torch.tensor(q, dtype=torch.float64).reshape(1, 1, 1, -1)
    kt = torch.tensor(k, dtype=torch.float64).reshape(1, 1, k.shape[0], -1)
    vt = torch.tensor(v, dtype=torch.float64).reshape(1, 1, v.shape[0], -1)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)
    return o.reshape(-1).numpy()


def _lossless_setup(rng, d=16, n=300, transform="identity"):
    L = d // 4
    books_k = rng.standard_normal((L, 256, 4)).astype(np.float16)
    books_v = rng.standard_normal((L, 256, 4)).astype(np.float16)
    # distinct codewords so every point has a unique nearest one
    for b in (books_k, books_v):
        for ell in range(L):
            _, idx = np.unique(b[ell].astype(np.float64), axis=0, return_index=True)
            assert idx.size == 256
    codes_k = rng.integers(0, 256, (n, L)).astype(np.uint8)
    codes_v = rng.integers(0, 256, (n, L)).astype(np.uint8)
    r = vq.lookup(codes_k, books_k)
    s = vq.lookup(codes_v, books_v)
    if transform == "identity":
        t_k = np.eye(d)
        t_v = np.eye(d)
        kbar = np.zeros(d)
    else:
        t_k = rng.standard_normal((d, d)) + 3 * np.eye(d)
        t_v, _ = np.linalg.qr(rng.standard_normal((d, d)))
        kbar = rng.standard_normal(d)
    t_k_inv_t = np.linalg.inv(t_k).T
    k = r @ np.linalg.inv(t_k) + kbar          # keys whose coefficients are exactly codewords
    v = s @ np.linalg.inv(t_v)
    params = {"kbar": kbar, "t_k": t_k, "t_k_inv_t": t_k_inv_t, "t_v": t_v,
              "cb_k": books_k, "cb_v": books_v}
    return params, k, v, codes_k, codes_v


@pytest.mark.parametrize("transform", ["identity", "general"])
def test_lossless_codes_reduce_to_exact_attention(transform):
    """Identity (or any exact) transform + lossless codebooks: exact softmax attention."""
    rng = np.random.default_rng(0 if transform == "identity" else 1)
    d = 16
    params, k, v, ck_true, cv_true = _lossless_setup(rng, d=d, transform=transform)
    ck, gk, cv, gv = codec.encode_tokens(k, v, params)
    assert np.array_equal(ck, ck_true) and np.array_equal(cv, cv_true)
    scale = 1 / np.sqrt(d)
    for _ in range(3):
        q = rng.standard_normal(d) * 2
        out = att.decode_row(q, ck, cv, params, scale)
        assert np.allclose(out, _sdpa(q, k, v, scale), atol=1e-10)


def test_sink_is_a_valueless_extra_logit():
    """A sink logit s equals an extra key with q.k*scale = s and a zero value."""
    rng = np.random.default_rng(2)
    d = 16
    params, k, v, ck, cv = _lossless_setup(rng, d=d, transform="general")
    scale = 1 / np.sqrt(d)
    q = rng.standard_normal(d)
    s = 0.7
    k_sink = q * (s / (scale * (q @ q)))
    ref = _sdpa(q, np.vstack([k, k_sink]), np.vstack([v, np.zeros(d)]), scale)
    out = att.decode_row(q, ck, cv, params, scale, sink=s)
    assert np.allclose(out, ref, atol=1e-10)


def test_window_and_empty():
    rng = np.random.default_rng(3)
    d = 16
    params, k, v, ck, cv = _lossless_setup(rng, d=d, transform="general", n=50)
    scale = 0.25
    q = rng.standard_normal(d)
    full = att.decode_row(q, ck, cv, params, scale)
    assert np.allclose(att.decode_row(q, ck, cv, params, scale, window=500), full, atol=1e-13)
    assert np.allclose(att.decode_row(q, ck, cv, params, scale, window=1), v[-1], atol=1e-10)
    assert np.allclose(att.decode_row(q, ck, cv, params, scale, window=7),
                       _sdpa(q, k[-7:], v[-7:], scale), atol=1e-10)
    empty = ck[:0]
    assert np.all(att.decode_row(q, empty, empty, params, scale) == 0)
    assert np.all(att.decode_row(q, empty, empty, params, scale, sink=1.0) == 0)


def test_offset_invariance_lemma_s1():
    """Lemma S1: a common key offset leaves attention unchanged -- unless a sink is present."""
    rng = np.random.default_rng(4)
    d = 16
    params, k, v, ck, cv = _lossless_setup(rng, d=d, transform="general")
    scale = 1 / np.sqrt(d)
    q = rng.standard_normal(d)
    shifted = dict(params)
    c = rng.standard_normal(d) * 3
    shifted["kbar"] = params["kbar"] + c
    a = att.decode_row(q, ck, cv, params, scale)
    b = att.decode_row(q, ck, cv, shifted, scale)
    assert np.allclose(a, b, atol=1e-12)
    a_s = att.decode_row(q, ck, cv, params, scale, sink=0.3)
    b_s = att.decode_row(q, ck, cv, shifted, scale, sink=0.3)
    assert not np.allclose(a_s, b_s, atol=1e-6)
    # shifting the sink by the same per-query constant restores equality
    b_fix = att.decode_row(q, ck, cv, shifted, scale, sink=0.3 + (q @ c) * scale)
    assert np.allclose(a_s, b_fix, atol=1e-12)


@pytest.mark.parametrize("n_split", [1, 2, 7, 64])
@pytest.mark.parametrize("window,sink", [(0, None), (0, -0.4), (33, 1.2), (1000, None)])
def test_fast_form_equals_plain_form(n_split, window, sink):
    """q' = q R_K^{-T} * scale, k_bar dropped, shifted sink, split merge: equal to plain form."""
    rng = np.random.default_rng(5)
    d = 32
    L = d // 4
    params = {
        "kbar": rng.standard_normal(d).astype(np.float32),
        "t_k": rng.standard_normal((d, d)).astype(np.float32),
        "t_k_inv_t": rng.standard_normal((d, d)).astype(np.float32),
        "t_v": rng.standard_normal((d, d)).astype(np.float32),
        "cb_k": rng.standard_normal((L, 256, 4)).astype(np.float16),
        "cb_v": rng.standard_normal((L, 256, 4)).astype(np.float16),
    }
    ck = rng.integers(0, 256, (400, L)).astype(np.uint8)
    cv = rng.integers(0, 256, (400, L)).astype(np.uint8)
    q = rng.standard_normal(d)
    scale = 1 / np.sqrt(d)
    plain = att.decode_row(q, ck, cv, params, scale, window, sink)
    fast = att.decode_row_fast(q, ck, cv, params, scale, window, sink, n_split)
    assert np.allclose(plain, fast, rtol=1e-12, atol=1e-12 * np.abs(plain).max())
