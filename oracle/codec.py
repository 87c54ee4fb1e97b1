"""Oracle append-time encoder (write path).

Test infrastructure only (see ``oracle/__init__.py``).

Paper, Algorithm 1 (inference, write) and Theorem 1: a key is centred and
transformed, r = (k - k_bar) R_K, and each group of g coefficients is replaced
by the index of its nearest codeword; values are transformed by R_V
(Corollary 1, s = v R_V) and encoded the same way.  All arithmetic in fp64 on
the stored fp32 transforms and mean and the stored fp16 codebooks.

Key-scale format (Algorithm 2's normalization; Sec. "Bit rate": a BF16 scale
per token; Sec. "Decoding kernel and read path": the read path multiplies the
partial logit by it): rho = ||r||_2 / sqrt(d) and the codes quantize r / rho
against codebooks trained on normalized coefficients.  Readings fixed here:
||r||^2 is summed in coordinate order with each square rounded; rho =
sqrt(||r||^2) / sqrt(d); the stored scale is rho rounded to fp32 and then to
bf16 (both to nearest even), and the decode uses the stored value; a key with
r = 0 gets rho = 0 and the codes of the zero vector.
"""

from __future__ import annotations

import numpy as np

from .vq import encode


def key_coefficients(k: np.ndarray, kbar: np.ndarray, t_k: np.ndarray) -> np.ndarray:
    """r = (k - k_bar) t_k for every row of k (n, D)."""
    return (np.asarray(k, dtype=np.float64) - np.asarray(kbar, dtype=np.float64)) @ \
        np.asarray(t_k, dtype=np.float64)


def value_coefficients(v: np.ndarray, t_v: np.ndarray) -> np.ndarray:
    """s = v t_v for every row of v (n, D)."""
    return np.asarray(v, dtype=np.float64) @ np.asarray(t_v, dtype=np.float64)


def key_scale(r: np.ndarray) -> np.ndarray:
    """rho = ||r||_2 / sqrt(d) per row of r (n, d), in fp64 (Algorithm 2)."""
    r = np.asarray(r, dtype=np.float64)
    ss = np.cumsum(r * r, axis=-1)[..., -1]  # sequential sum of the rounded squares
    return np.sqrt(ss) / np.sqrt(float(r.shape[-1]))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Stored bf16 bit patterns of fp64 values: to fp32, then to bf16, each to nearest even."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def bf16_value(bits: np.ndarray) -> np.ndarray:
    """fp64 value of bf16 bit patterns."""
    return (np.asarray(bits, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)


def band_values(x: np.ndarray) -> np.ndarray:
    """Exact rows of the sink-plus-recent band: the inputs as stored in BF16 (fp64 values)."""
    return bf16_value(bf16_bits(x))


def normalized_key_coefficients(r: np.ndarray):
    """(r / rho, rho) with rows of r = 0 mapped to (0, 0)."""
    rho = key_scale(r)
    safe = np.where(rho > 0.0, rho, 1.0)
    rn = np.where(rho[:, None] > 0.0, np.asarray(r, dtype=np.float64) / safe[:, None], 0.0)
    return rn, rho


def encode_tokens_scaled(k: np.ndarray, v: np.ndarray, params_head: dict):
    """Key-scale format: codes and near-tie gaps of n keys and values (n, D) and the keys' stored scales.

    Returns (codes_k, gap_k, scale_bits, codes_v, gap_v, rho) where scale_bits
    are the stored bf16 patterns (n,) and rho the fp64 scales before storage.
    """
    r = key_coefficients(k, params_head["kbar"], params_head["t_k"])
    rn, rho = normalized_key_coefficients(r)
    ck, gk = encode(rn, params_head["cb_k"])
    cv, gv = encode(value_coefficients(v, params_head["t_v"]), params_head["cb_v"])
    return ck, gk, bf16_bits(rho), cv, gv, rho


# ---------------------------------------------------------------------------
# Scalar value arm (paper: Sec. "Bit rate": INT2 values with a BF16 scale and
# offset per token; the implementation table: per-token affine INT2; Sec.
# "Decoding kernel and read path": dequantized in the rotation basis whose
# inverse is applied after the attention sum).  The rotation is the stored
# value transform t_v (any orthogonal matrix: R_V, or a Hadamard rotation).
# Readings fixed here: min-max affine grid over the D coordinates of a token,
# offset = bf16(min), scale = bf16((max - min) / 3) (fp64 arithmetic, each
# rounded to fp32 then to bf16, to nearest even); the codes use the stored
# offset and scale: q_i = clamp(round_half_even((s_i - offset) / scale), 0, 3),
# all codes 0 when the stored scale is 0; coordinate 4g + j of a token is
# stored in bits 2j, 2j + 1 of its byte g.
# ---------------------------------------------------------------------------

def sq_encode_values(v: np.ndarray, t_v: np.ndarray):
    """Per-token affine INT2 of s = v t_v: (packed bytes (n, D/4) uint8, scale bits (n,), offset bits (n,))."""
    s = value_coefficients(v, t_v)
    mn = s.min(axis=1)
    mx = s.max(axis=1)
    zero_bits = bf16_bits(mn)
    scale_bits = bf16_bits((mx - mn) / 3.0)
    zero = bf16_value(zero_bits)[:, None]
    scale = bf16_value(scale_bits)[:, None]
    safe = np.where(scale > 0, scale, 1.0)
    q = np.where(scale > 0, np.clip(np.rint((s - zero) / safe), 0, 3), 0).astype(np.uint8)
    n, d = q.shape
    qg = q.reshape(n, d // 4, 4)
    packed = (qg[..., 0] | (qg[..., 1] << 2) | (qg[..., 2] << 4) | (qg[..., 3] << 6)).astype(np.uint8)
    return packed, scale_bits, zero_bits


def sq_unpack(packed: np.ndarray) -> np.ndarray:
    """INT2 codes (n, D) of packed bytes (n, D/4)."""
    p = np.asarray(packed, dtype=np.uint8)
    q = np.stack([(p >> (2 * j)) & 3 for j in range(4)], axis=-1)
    return q.reshape(p.shape[0], 4 * p.shape[1])


def sq_reconstruct(packed: np.ndarray, scale_bits: np.ndarray, zero_bits: np.ndarray) -> np.ndarray:
    """s_hat = offset + scale * q per token (rotation basis), fp64."""
    q = sq_unpack(packed).astype(np.float64)
    return bf16_value(zero_bits)[:, None] + bf16_value(scale_bits)[:, None] * q


def encode_tokens(k: np.ndarray, v: np.ndarray, params_head: dict):
    """Codes and near-tie gaps of n keys and values (n, D) of one KV head.

    Returns (codes_k, gap_k, codes_v, gap_v); codes are uint8 (n, L).
    """
    ck, gk = encode(key_coefficients(k, params_head["kbar"], params_head["t_k"]),
                    params_head["cb_k"])
    cv, gv = encode(value_coefficients(v, params_head["t_v"]), params_head["cb_v"])
    return ck, gk, cv, gv
