"""Oracle append-time encoder (write path).

Test infrastructure only (see ``oracle/__init__.py``).

Paper, Algorithm 1 (inference, write) and Theorem 1: a key is centred and
transformed, r = (k - k_bar) R_K, and each group of g coefficients is replaced
by the index of its nearest codeword; values are transformed by R_V
(Corollary 1, s = v R_V) and encoded the same way.  All arithmetic in fp64 on
the stored fp32 transforms and mean and the stored fp16 codebooks.
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


def encode_tokens(k: np.ndarray, v: np.ndarray, params_head: dict):
    """Codes and near-tie gaps of n keys and values (n, D) of one KV head.

    Returns (codes_k, gap_k, codes_v, gap_v); codes are uint8 (n, L).
    """
    ck, gk = encode(key_coefficients(k, params_head["kbar"], params_head["t_k"]),
                    params_head["cb_k"])
    cv, gv = encode(value_coefficients(v, params_head["t_v"]), params_head["cb_v"])
    return ck, gk, cv, gv
