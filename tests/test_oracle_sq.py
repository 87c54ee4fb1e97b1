"""Pins for the oracle's scalar value arm (per-token affine INT2 in a rotation basis)."""

import numpy as np
import torch

from oracle import attention as att
from oracle import codec


def _hadamard(d):
    h = np.array([[1.0]])
    while h.shape[0] < d:
        h = np.block([[h, h], [h, -h]])
    return h / np.sqrt(d)


def test_packing_layout():
    # codes of coordinates 0..7 of one token: byte g holds coordinate 4g + j in bits 2j, 2j+1
    s = np.array([[0.0, 1.0, 2.0, 3.0, 3.0, 2.0, 1.0, 0.0]])
    packed, sb, zb = codec.sq_encode_values(s, np.eye(8))
    assert codec.bf16_value(zb)[0] == 0.0 and codec.bf16_value(sb)[0] == 1.0
    assert packed.tolist() == [[0xE4, 0x1B]]
    assert codec.sq_unpack(packed).tolist() == [[0, 1, 2, 3, 3, 2, 1, 0]]


def test_rows_on_the_grid_are_exact():
    rng = np.random.default_rng(1)
    for _ in range(20):
        a = float(codec.bf16_value(codec.bf16_bits(np.array([rng.normal() * 4])))[0])
        h = 2.0 ** int(rng.integers(-6, 3))
        q = rng.integers(0, 4, 64)
        q[:2] = [0, 3]                                   # min and max present
        s = (a + h * q)[None, :]
        packed, sb, zb = codec.sq_encode_values(s, np.eye(64))
        assert np.array_equal(codec.sq_unpack(packed)[0], q)
        assert np.array_equal(codec.sq_reconstruct(packed, sb, zb), s)


def test_constant_row_has_zero_scale():
    s = np.full((1, 16), 0.7)
    packed, sb, zb = codec.sq_encode_values(s, np.eye(16))
    assert int(sb[0]) == 0 and not packed.any()
    assert codec.sq_reconstruct(packed, sb, zb)[0, 0] == codec.bf16_value(codec.bf16_bits(np.array([0.7])))[0]


def test_error_bound_and_rotation():
    rng = np.random.default_rng(2)
    d = 64
    r = _hadamard(d)
    v = rng.standard_normal((300, d)) * np.exp(rng.uniform(-3, 3, (300, 1)))
    packed, sb, zb = codec.sq_encode_values(v, r)
    s = v @ r
    s_hat = codec.sq_reconstruct(packed, sb, zb)
    scale = codec.bf16_value(sb)
    mn = s.min(axis=1)
    bound = 0.5 * scale + 2.0 ** -8 * (np.abs(mn) + 3 * scale)
    assert np.all(np.abs(s - s_hat).max(axis=1) <= bound)
    # the rotation is orthogonal: the error norm is the same in both bases
    v_hat = att.reconstruct_values(packed, None, r, (sb, zb))
    assert np.allclose(np.linalg.norm(v - v_hat, axis=1), np.linalg.norm(s - s_hat, axis=1), rtol=1e-10)


def test_decode_is_attention_over_the_dequantized_values():
    rng = np.random.default_rng(3)
    d, n = 32, 120
    r = _hadamard(d)
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    # keys lossless: identity transforms and one exact codebook per group
    params = {"kbar": np.zeros(d), "t_k": np.eye(d), "t_k_inv_t": np.eye(d), "t_v": r,
              "cb_k": np.zeros((d // 4, 256, 4), dtype=np.float16), "cb_v": None}
    ck = np.zeros((n, d // 4), dtype=np.uint8)       # every key reconstructs to 0
    packed, sb, zb = codec.sq_encode_values(v, r)
    q = rng.standard_normal((2, d))
    out = att.decode_rows(q, ck, packed, params, 0.3, sq_v=(sb, zb))
    v_hat = codec.sq_reconstruct(packed, sb, zb) @ r.T
    # all logits equal (zero keys): the output is the mean of the dequantized values
    for h in range(2):
        qt = torch.tensor(q[h]).reshape(1, 1, 1, d)
        kt = torch.zeros((1, 1, n, d), dtype=torch.float64)
        vt = torch.tensor(v_hat).reshape(1, 1, n, d)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=0.3).reshape(-1).numpy()
        assert np.allclose(out[h], ref, rtol=1e-12, atol=1e-12)
        assert np.allclose(out[h], v_hat.mean(axis=0), rtol=1e-12, atol=1e-12)


def test_empty_rows():
    assert codec.sq_unpack(np.zeros((0, 8), dtype=np.uint8)).shape == (0, 32)
