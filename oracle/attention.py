"""Oracle decode attention over a NOVA-KV cache (plain and fast forms).

Test infrastructure only (see ``oracle/__init__.py``).  fp64 throughout.

Plain form -- the definition.  Reconstruct every attended key and value in the
original domain from its codes (paper, Sec. "Transform coding":
x_hat = Q(x R) R^{-1}; Theorem 1: k_hat = r_hat R_K^{-1} + k_bar; Corollary 1:
v_hat = s_hat R_V^T) and run textbook softmax attention (paper, Eq. "scores":
S = softmax(Q K^T / sqrt(d)), O = S V) for the single decode query.  A learned
sink (paper, Appendix "Attention sinks in the quantized serving path") is one
extra logit in the softmax with no value vector.

With stored t_k_inv_t = R_K^{-T}, R_K^{-1} = t_k_inv_t^T.

Readings: the window W attends to the last W cached tokens [S - W, S); a
sequence with no attended token and no sink yields a zero output.

Key-scale format (Algorithm 2's normalization, the read path's per-token
scale): the reconstructed key is k_hat = rho * Q(r/rho) R_K^{-1} + k_bar with
the stored (bf16) rho, so the logit of a token is rho times the logit of its
normalized code.

Sink-plus-recent band (Sec. "Sink-plus-recent band"; Fig. "Cache layout at
decoding position t"): the first n_sink and the most recent n_rec cached
positions are held exactly (BF16) instead of quantized; the attention runs
over all attended positions at once, band positions with their BF16 keys and
values, the others reconstructed from codes.  Readings: "most recent" is
positions [S - n_rec, S) of a sequence of S cached tokens; the band applies
inside the attended range (a window may cut it); band keys enter the logit as
they are (no k_bar shift in the plain form, which holds no shift at all).

Scalar value arm (Sec. "Bit rate"; implementation table: per-token affine
INT2 values): v_hat = (offset + scale * q) t_v^T with the stored bf16 offset
and scale of the token (oracle/codec.py holds the encoder).

Fast form -- for self-consistency only (Algorithm 1 inference step; Sec.
"Decoding kernel and read path"; sinks appendix): q' = q R_K^{-T} * scale,
logit = q' . r_hat (k_bar dropped, Lemma S1), sink shifted by -(q . k_bar) * scale,
any number of context splits merged by log-sum-exp, sink added once after the
merge, value accumulated in the transform domain and mapped back by t_v^T once.
"""

from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from .codec import sq_reconstruct
from .vq import lookup


def attended_range(seq_len: int, window: int):
    lo = max(0, seq_len - window) if window > 0 else 0
    return lo, seq_len


def band_mask(seq_len: int, n_sink: int, n_rec: int) -> np.ndarray:
    """Positions of a sequence of seq_len tokens held exactly: t < n_sink or t >= seq_len - n_rec."""
    t = np.arange(seq_len)
    return (t < n_sink) | (t >= seq_len - n_rec)


def _with_band(k_hat, v_hat, lo, hi, band):
    """Replace the band positions of the attended rows [lo, hi) by their exact rows."""
    if band is None:
        return k_hat, v_hat
    n_sink, n_rec, k_exact, v_exact = band
    m = band_mask(hi, n_sink, n_rec)[lo:hi]
    k_hat = k_hat.copy()
    v_hat = v_hat.copy()
    k_hat[m] = np.asarray(k_exact, dtype=np.float64)[lo:hi][m]
    v_hat[m] = np.asarray(v_exact, dtype=np.float64)[lo:hi][m]
    return k_hat, v_hat


def reconstruct_keys(codes_k: np.ndarray, cb_k: np.ndarray, t_k_inv_t: np.ndarray,
                     kbar: np.ndarray, scales: Optional[np.ndarray] = None) -> np.ndarray:
    """k_hat = Q(r) R_K^{-1} + k_bar for every row of codes (n, L); with per-token
    scales (n,) (key-scale format) k_hat = rho * Q(r/rho) R_K^{-1} + k_bar."""
    r_hat = lookup(codes_k, cb_k)
    if scales is not None:
        r_hat = r_hat * np.asarray(scales, dtype=np.float64)[:, None]
    return r_hat @ np.asarray(t_k_inv_t, dtype=np.float64).T + np.asarray(kbar, dtype=np.float64)


def reconstruct_values(codes_v: np.ndarray, cb_v: np.ndarray, t_v: np.ndarray, sq=None) -> np.ndarray:
    """v_hat = Q(s) R_V^T for every row of codes (n, L).  With sq = (scale bits
    (n,), offset bits (n,)) the codes are the scalar value arm's packed INT2
    and Q(s) = offset + scale * q (cb_v unused)."""
    if sq is not None:
        s_hat = sq_reconstruct(codes_v, sq[0], sq[1])
    else:
        s_hat = lookup(codes_v, cb_v)
    return s_hat @ np.asarray(t_v, dtype=np.float64).T


def softmax_attention(q: np.ndarray, keys: np.ndarray, values: np.ndarray, scale: float,
                      sink: Optional[float] = None) -> np.ndarray:
    """Textbook single-query softmax attention with an optional value-less sink logit."""
    z = (keys @ np.asarray(q, dtype=np.float64)) * scale
    if sink is not None:
        zall = np.concatenate([z, [float(sink)]])
    else:
        zall = z
    if zall.size == 0:
        return np.zeros(values.shape[1])
    m = zall.max()
    e = np.exp(zall - m)
    denom = e.sum()
    return (e[:z.size] @ values) / denom


def decode_row(q: np.ndarray, codes_k: np.ndarray, codes_v: np.ndarray, params_head: dict,
               scale: float, window: int = 0, sink: Optional[float] = None,
               scales_k: Optional[np.ndarray] = None, band=None) -> np.ndarray:
    """Plain-form output of one query head over one sequence's cached codes (S, L);
    scales_k (S,) are the stored per-token key scales of the key-scale format;
    band = (n_sink, n_rec, k_exact (S, D), v_exact (S, D)) holds the exact
    rows of the sink-plus-recent band (rows outside it are not read)."""
    lo, hi = attended_range(codes_k.shape[0], window)
    k_hat = reconstruct_keys(codes_k[lo:hi], params_head["cb_k"], params_head["t_k_inv_t"],
                             params_head["kbar"], None if scales_k is None else scales_k[lo:hi])
    v_hat = reconstruct_values(codes_v[lo:hi], params_head["cb_v"], params_head["t_v"])
    k_hat, v_hat = _with_band(k_hat, v_hat, lo, hi, band)
    return softmax_attention(q, k_hat, v_hat, scale, sink)


def decode_rows(q_heads: np.ndarray, codes_k: np.ndarray, codes_v: np.ndarray,
                params_head: dict, scale: float, window: int = 0,
                sinks: Optional[Sequence[float]] = None,
                scales_k: Optional[np.ndarray] = None, band=None, sq_v=None) -> np.ndarray:
    """Plain-form outputs of the G query heads sharing one KV head: q_heads (G, D) -> (G, D).
    band as in decode_row; sq_v = (scale bits (S,), offset bits (S,)) for the
    scalar value arm (codes_v then holds packed INT2, (S, D/4))."""
    lo, hi = attended_range(codes_k.shape[0], window)
    k_hat = reconstruct_keys(codes_k[lo:hi], params_head["cb_k"], params_head["t_k_inv_t"],
                             params_head["kbar"], None if scales_k is None else scales_k[lo:hi])
    v_hat = reconstruct_values(codes_v[lo:hi], params_head.get("cb_v"), params_head["t_v"],
                               None if sq_v is None else (sq_v[0][lo:hi], sq_v[1][lo:hi]))
    k_hat, v_hat = _with_band(k_hat, v_hat, lo, hi, band)
    out = np.empty((q_heads.shape[0], v_hat.shape[1]))
    for h in range(q_heads.shape[0]):
        out[h] = softmax_attention(q_heads[h], k_hat, v_hat, scale,
                                   None if sinks is None else sinks[h])
    return out


def decode_row_fast(q: np.ndarray, codes_k: np.ndarray, codes_v: np.ndarray, params_head: dict,
                    scale: float, window: int = 0, sink: Optional[float] = None,
                    n_split: int = 1, scales_k: Optional[np.ndarray] = None) -> np.ndarray:
    """Fast (transform-domain, split-context) form of ``decode_row``; equal up to rounding."""
    lo, hi = attended_range(codes_k.shape[0], window)
    t_k_inv_t = np.asarray(params_head["t_k_inv_t"], dtype=np.float64)
    kbar = np.asarray(params_head["kbar"], dtype=np.float64)
    qp = (np.asarray(q, dtype=np.float64) @ t_k_inv_t) * scale
    r_hat = lookup(codes_k[lo:hi], params_head["cb_k"])
    s_hat = lookup(codes_v[lo:hi], params_head["cb_v"])
    z = r_hat @ qp
    if scales_k is not None:  # the read path's one multiply per token
        z = z * np.asarray(scales_k[lo:hi], dtype=np.float64)
    d = s_hat.shape[1]
    parts = []
    bounds = np.linspace(0, z.size, n_split + 1).astype(int)
    for a, b in zip(bounds[:-1], bounds[1:]):
        if b > a:
            m = z[a:b].max()
            e = np.exp(z[a:b] - m)
            parts.append((m, e.sum(), e @ s_hat[a:b]))
    shifted = None if sink is None else float(sink) - float(np.asarray(q, dtype=np.float64) @ kbar) * scale
    ms = [p[0] for p in parts] + ([shifted] if shifted is not None else [])
    if not ms:
        return np.zeros(d)
    big = max(ms)
    denom = sum(np.exp(m - big) * l for m, l, _ in parts)
    acc = sum((np.exp(m - big) * a for m, _, a in parts), np.zeros(d))
    if shifted is not None:
        denom += np.exp(shifted - big)
    s_out = acc / denom
    return s_out @ np.asarray(params_head["t_v"], dtype=np.float64).T


def head_params(params: dict, kv: int) -> dict:
    """Slice the [Hkv][...] stacked parameters down to one KV head."""
    return {k: v[kv] for k, v in params.items()}
