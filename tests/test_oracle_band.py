"""Pins for the oracle's sink-plus-recent band (first n_sink and last n_rec
positions held exactly in BF16, the rest quantized)."""

import numpy as np
import pytest
import torch

from oracle import attention as att
from oracle import codec


def _sdpa(q, k, v, scale):
    """Library reference: torch scaled_dot_product_attention in fp64 on the CPU."""
    qt = torch.tensor(q, dtype=torch.float64).reshape(1, 1, 1, -1)
    kt = torch.tensor(k, dtype=torch.float64).reshape(1, 1, k.shape[0], -1)
    vt = torch.tensor(v, dtype=torch.float64).reshape(1, 1, v.shape[0], -1)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)
    return o.reshape(-1).numpy()


def _setup(rng, d=16, n=200):
    """Random (lossy) parameters: an orthogonal t_v, a general t_k, random codebooks."""
    L = d // 4
    t_k = rng.standard_normal((d, d)) + 3 * np.eye(d)
    t_v, _ = np.linalg.qr(rng.standard_normal((d, d)))
    params = {"kbar": 0.3 * rng.standard_normal(d), "t_k": t_k, "t_k_inv_t": np.linalg.inv(t_k).T,
              "t_v": t_v, "cb_k": rng.standard_normal((L, 256, 4)).astype(np.float16),
              "cb_v": rng.standard_normal((L, 256, 4)).astype(np.float16)}
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    ck, _, cv, _ = codec.encode_tokens(k, v, params)
    return params, k, v, ck, cv


def test_band_mask_closed_forms():
    assert np.flatnonzero(att.band_mask(10, 2, 3)).tolist() == [0, 1, 7, 8, 9]
    assert att.band_mask(4, 2, 3).all()                 # the band covers a short sequence
    assert not att.band_mask(6, 0, 0).any()
    assert np.flatnonzero(att.band_mask(6, 0, 2)).tolist() == [4, 5]
    assert np.flatnonzero(att.band_mask(6, 3, 0)).tolist() == [0, 1, 2]
    assert att.band_mask(0, 64, 256).size == 0


def test_band_values_are_bf16_roundings():
    x = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -3.14159, 0.0])
    assert codec.band_values(x).tolist() == [1.0, 1.0, 1.0 + 2.0 ** -6, -3.140625, 0.0]


def test_band_over_the_whole_sequence_is_exact_attention():
    """n_sink + n_rec >= S: every key and value is the BF16 input, so the output is
    textbook attention over them (library SDPA), whatever the codes."""
    rng = np.random.default_rng(5)
    d, n = 16, 40
    params, k, v, ck, cv = _setup(rng, d, n)
    kb, vb = codec.band_values(k), codec.band_values(v)
    scale = 1 / np.sqrt(d)
    q = rng.standard_normal((3, d))
    for n_sink, n_rec in [(40, 0), (0, 40), (16, 24), (30, 30)]:
        out = att.decode_rows(q, ck, cv, params, scale, band=(n_sink, n_rec, kb, vb))
        for h in range(3):
            assert np.allclose(out[h], _sdpa(q[h], kb, vb, scale), rtol=1e-12, atol=1e-12)


def test_empty_band_is_the_plain_decode():
    rng = np.random.default_rng(6)
    params, k, v, ck, cv = _setup(rng)
    q = rng.standard_normal((2, 16))
    a = att.decode_rows(q, ck, cv, params, 0.25)
    b = att.decode_rows(q, ck, cv, params, 0.25, band=(0, 0, k, v))
    assert np.array_equal(a, b)


@pytest.mark.parametrize("window", [0, 50, 150])
def test_band_mixes_exact_and_reconstructed_rows(window):
    """Brute force: the attention over the row set {exact rows at band positions,
    reconstructed rows elsewhere} of the attended range, with a sink."""
    rng = np.random.default_rng(7)
    d, n = 16, 200
    params, k, v, ck, cv = _setup(rng, d, n)
    kb, vb = codec.band_values(k), codec.band_values(v)
    n_sink, n_rec = 8, 32
    scale = 1 / np.sqrt(d)
    q = rng.standard_normal(d)
    sink = 0.7
    out = att.decode_row(q, ck, cv, params, scale, window=window, sink=sink, band=(n_sink, n_rec, kb, vb))
    lo = n - window if window else 0
    rows_k, rows_v = [], []
    for t in range(lo, n):
        if t < n_sink or t >= n - n_rec:
            rows_k.append(kb[t])
            rows_v.append(vb[t])
        else:
            rows_k.append(att.reconstruct_keys(ck[t:t + 1], params["cb_k"], params["t_k_inv_t"], params["kbar"])[0])
            rows_v.append(att.reconstruct_values(cv[t:t + 1], params["cb_v"], params["t_v"])[0])
    z = np.array([q @ r for r in rows_k]) * scale
    w = np.exp(np.concatenate([z, [sink]]) - max(z.max(), sink))
    ref = (w[:-1] @ np.array(rows_v)) / w.sum()
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-13)
    # the band changes the output (the quantization is lossy)
    plain = att.decode_row(q, ck, cv, params, scale, window=window, sink=sink)
    assert not np.allclose(out, plain, rtol=1e-6, atol=1e-9)


def test_band_rows_outside_the_band_are_never_read():
    rng = np.random.default_rng(8)
    params, k, v, ck, cv = _setup(rng, 16, 100)
    kb, vb = codec.band_values(k), codec.band_values(v)
    m = att.band_mask(100, 4, 10)
    kn, vn = kb.copy(), vb.copy()
    kn[~m] = np.nan
    vn[~m] = np.nan
    q = rng.standard_normal((2, 16))
    a = att.decode_rows(q, ck, cv, params, 0.25, band=(4, 10, kb, vb))
    b = att.decode_rows(q, ck, cv, params, 0.25, band=(4, 10, kn, vn))
    assert np.array_equal(a, b)
