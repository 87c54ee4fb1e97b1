"""Pins for the oracle's key-scale format (per-token key scale rho = ||r|| / sqrt(d)).

Paper: Algorithm 2 (normalize r_j by rho_j before the codebooks are trained),
Sec. "Bit rate" (one BF16 scale per token on the K side), Sec. "Decoding kernel
and read path" (the read path multiplies the partial logit by rho_j).
"""

import numpy as np
import pytest

from oracle import attention as att
from oracle import calibration, codec, vq


def test_key_scale_closed_forms():
    d = 128
    assert codec.key_scale(np.ones((1, d)))[0] == 1.0            # ||1|| = sqrt(d)
    assert codec.key_scale(2.0 * np.ones((1, d)))[0] == 2.0
    r = np.zeros((1, 4))
    r[0, 0], r[0, 1] = 3.0, 4.0
    assert codec.key_scale(r)[0] == 2.5                          # 5 / sqrt(4)
    assert codec.key_scale(np.zeros((2, 16))).tolist() == [0.0, 0.0]


def test_bf16_storage_rounds_to_fp32_then_to_bf16():
    one = 1.0
    cases = {
        one: 0x3F80,
        one + 2.0 ** -8: 0x3F80,                  # tie -> even
        one + 3 * 2.0 ** -8: 0x3F82,              # tie -> even (upward)
        one + 2.0 ** -8 + 2.0 ** -20: 0x3F81,     # above the tie
        # fp32 rounding first drops 2^-30, leaving the tie, which goes to even;
        # a single rounding from fp64 would give 0x3F81
        one + 2.0 ** -8 + 2.0 ** -30: 0x3F80,
        0.0: 0x0000,
        -2.0: 0xC000,
    }
    for x, bits in cases.items():
        assert int(codec.bf16_bits(np.array([x]))[0]) == bits, (x, hex(bits))
        assert codec.bf16_value(np.array([bits], dtype=np.uint16))[0] == np.float64(np.float32(
            np.frombuffer(np.uint32(bits << 16).tobytes(), dtype=np.float32)[0]))


def test_normalization_is_scale_invariant_and_has_unit_rms():
    rng = np.random.default_rng(11)
    r = rng.standard_normal((200, 128)) * rng.uniform(0.1, 10.0, (200, 1))
    rn, rho = codec.normalized_key_coefficients(r)
    rn2, rho2 = codec.normalized_key_coefficients(2.0 * r)       # exact power-of-two scaling
    assert np.array_equal(rn, rn2) and np.array_equal(rho2, 2.0 * rho)
    rms = np.sqrt((rn * rn).mean(axis=1))
    assert np.allclose(rms, 1.0, rtol=1e-14, atol=0)
    z, rz = codec.normalized_key_coefficients(np.zeros((1, 128)))
    assert rz[0] == 0.0 and not z.any()


def _scaled_params(rng, d=32, m=4000):
    """Calibrated parameters of the key-scale format on anisotropic synthetic keys."""
    spec = np.exp(-np.arange(d) / 6.0) + 0.05
    k_cal = rng.standard_normal((m, d)) * spec * rng.uniform(0.3, 3.0, (m, 1)) + 0.5
    v_cal = rng.standard_normal((m, d)) * spec[::-1]
    q_cal = rng.standard_normal((2, m, d)) * spec
    stored, _ = calibration.calibrate_head(k_cal, v_cal, q_cal, kmeans_iters=8, seed=3, key_scale=True,
                                           mo_stride=64)
    return stored, k_cal, v_cal


def test_scaled_codebooks_are_trained_on_normalized_coefficients():
    rng = np.random.default_rng(5)
    stored, k_cal, _ = _scaled_params(rng)
    cb = stored["cb_k"].astype(np.float64)
    # normalized coefficients have mean square 1 per coordinate summed over the
    # vector, so the codewords' mean squared norm is close to g (= 4) times 1
    msq = (cb * cb).sum(axis=2).mean()
    assert 1.0 < msq < 6.0, msq
    unscaled, _ = calibration.calibrate_head(k_cal, k_cal[::-1], np.stack([k_cal, k_cal]), kmeans_iters=2,
                                             seed=3, mo_stride=256)
    assert not np.array_equal(unscaled["cb_k"], stored["cb_k"])


def test_scaled_reconstruction_and_attention_are_within_the_quantization_error():
    """The scale multiplies the normalized codeword back: k_hat tracks k, and the
    decode output tracks exact attention over the original keys."""
    rng = np.random.default_rng(7)
    d = 32
    stored, k_cal, v_cal = _scaled_params(rng, d=d)
    p = {k: np.asarray(v) for k, v in stored.items()}
    k = k_cal[:600]
    v = v_cal[:600]
    ck, gk, sbits, cv, gv, rho = codec.encode_tokens_scaled(k, v, p)
    scales = codec.bf16_value(sbits)
    assert np.allclose(scales, rho, rtol=2.0 ** -8, atol=0)
    k_hat = att.reconstruct_keys(ck, p["cb_k"], p["t_k_inv_t"], p["kbar"], scales)
    rel = np.linalg.norm(k_hat - k, axis=1) / np.linalg.norm(k - p["kbar"].astype(np.float64), axis=1)
    assert np.median(rel) < 0.35, np.median(rel)
    # the same keys without their scales are far off: the scale is not cosmetic
    k_noscale = att.reconstruct_keys(ck, p["cb_k"], p["t_k_inv_t"], p["kbar"])
    rel_noscale = np.linalg.norm(k_noscale - k, axis=1) / np.linalg.norm(k - p["kbar"].astype(np.float64), axis=1)
    assert np.median(rel_noscale) > 2 * np.median(rel)
    scale = 1 / np.sqrt(d)
    q = rng.standard_normal(d)
    exact = att.softmax_attention(q, k, v, scale)
    got = att.decode_row(q, ck, cv, p, scale, scales_k=scales)
    assert np.linalg.norm(got - exact) < 0.25 * np.linalg.norm(exact)


def test_unit_scales_reduce_to_the_unscaled_decode():
    rng = np.random.default_rng(9)
    d, n = 16, 50
    L = d // 4
    p = {"kbar": rng.standard_normal(d), "t_k": np.eye(d), "t_k_inv_t": np.eye(d), "t_v": np.eye(d),
         "cb_k": rng.standard_normal((L, 256, 4)).astype(np.float16),
         "cb_v": rng.standard_normal((L, 256, 4)).astype(np.float16)}
    ck = rng.integers(0, 256, (n, L)).astype(np.uint8)
    cv = rng.integers(0, 256, (n, L)).astype(np.uint8)
    q = rng.standard_normal(d)
    a = att.decode_row(q, ck, cv, p, 0.25, window=20, sink=0.3)
    b = att.decode_row(q, ck, cv, p, 0.25, window=20, sink=0.3, scales_k=np.ones(n))
    assert np.array_equal(a, b)


@pytest.mark.parametrize("n_split", [1, 3])
def test_scaled_fast_form_matches_plain_form(n_split):
    rng = np.random.default_rng(13)
    d, n = 16, 90
    L = d // 4
    t_k = rng.standard_normal((d, d)) + 3 * np.eye(d)
    t_v, _ = np.linalg.qr(rng.standard_normal((d, d)))
    p = {"kbar": rng.standard_normal(d), "t_k": t_k, "t_k_inv_t": np.linalg.inv(t_k).T, "t_v": t_v,
         "cb_k": rng.standard_normal((L, 256, 4)).astype(np.float16),
         "cb_v": rng.standard_normal((L, 256, 4)).astype(np.float16)}
    ck = rng.integers(0, 256, (n, L)).astype(np.uint8)
    cv = rng.integers(0, 256, (n, L)).astype(np.uint8)
    scales = codec.bf16_value(codec.bf16_bits(rng.uniform(0.2, 3.0, n)))
    q = rng.standard_normal(d)
    plain = att.decode_row(q, ck, cv, p, 0.3, window=60, sink=0.5, scales_k=scales)
    fast = att.decode_row_fast(q, ck, cv, p, 0.3, window=60, sink=0.5, n_split=n_split, scales_k=scales)
    assert np.allclose(plain, fast, rtol=1e-11, atol=1e-12)
    # a single attended token: the output is its value whatever its scale
    one = att.decode_row(q, ck[:1], cv[:1], p, 0.3, scales_k=np.array([7.0]))
    assert np.allclose(one, vq.lookup(cv[:1], p["cb_v"])[0] @ t_v.T, rtol=1e-12, atol=1e-12)
