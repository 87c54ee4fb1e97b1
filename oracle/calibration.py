"""Oracle calibration: statistics, closed-form transforms, grouping fold, codebooks.

Test infrastructure only (see ``oracle/__init__.py``).  Plain fp64 NumPy,
written step by step from the paper:

* Algorithm 2 / Theorem 1 -- key transform R_K = M_q^{1/2} E and R_K^{-T} = M_q^{-1/2} E,
  E the eigenvectors of M_q^{1/2} S_k M_q^{1/2};
* Appendix "Query statistics under GQA" -- M_q summed over the query heads of a KV head;
* Corollary 1 -- value transform R_V = eigenvectors of M_o = sum_i o_i^T o_i;
* Theorem 2 / Sec. "KV cache vector quantization" -- volume-equalizing grouping,
  coordinate of rank r dealt to group r mod L, folded into the transform columns;
* Algorithm 3 -- one k-means codebook per group.

Readings where the paper is silent or loose (each also listed in the design notes):
* M_q, S_k and M_o are means rather than sums (divided by the number of
  terms).  Theorem 1 fixes R_K only through U U^T = c M_q, so a global scale
  leaves codes and logits unchanged; the mean keeps coefficients at logit scale.
* Eigenvalues in decreasing order; each eigenvector's largest-magnitude entry
  is made positive.
* Within group l the coordinate of rank r sits at slot floor(r / L), i.e. at
  column (r mod L) * g + floor(r / L) of the folded transform.
* Values are grouped by the empirical variance of v R_V on the calibration set.
* M_o uses causal attention of every ``mo_stride``-th calibration position
  over the calibration prefix (prefill statistics).
"""

from __future__ import annotations

import numpy as np

from .codec import normalized_key_coefficients
from .vq import train_codebooks

EIG_FLOOR = 1e-30


def query_second_moment(q_heads: np.ndarray) -> np.ndarray:
    """M_q for one KV head from calibration queries q_heads (G, M, D).

    Paper, Algorithm 2 first step and Appendix "Query statistics under GQA":
    M_q = sum_h sum_j q_j^(h)T q_j^(h).  Here divided by G*M (mean).
    """
    g, m, d = q_heads.shape
    mq = np.zeros((d, d))
    for h in range(g):
        mq += q_heads[h].T @ q_heads[h]
    return mq / (g * m)


def key_statistics(k: np.ndarray):
    """Key mean k_bar and centred scatter S_k = sum_j (k_j - k_bar)^T (k_j - k_bar) / M.

    Paper, Algorithm 2 second step (divided by M).
    """
    m = k.shape[0]
    kbar = k.mean(axis=0)
    kc = k - kbar
    return kbar, (kc.T @ kc) / m


def sym_power(mat: np.ndarray, p: float, floor: float = EIG_FLOOR) -> np.ndarray:
    """Symmetric power of a PSD matrix via its eigendecomposition, eigenvalues floored.

    Paper, Appendix "Calibration statistics" / "Calibration": M_q^{+-1/2} from the
    symmetric eigendecomposition with eigenvalues floored at 1e-30, no ridge.
    """
    w, u = np.linalg.eigh(0.5 * (mat + mat.T))
    w = np.maximum(w, floor)
    return (u * w ** p) @ u.T


def eig_descending(mat: np.ndarray):
    """Eigenpairs of a symmetric matrix, eigenvalues decreasing, sign-normalised columns."""
    w, e = np.linalg.eigh(0.5 * (mat + mat.T))
    order = np.argsort(w)[::-1]
    w = w[order]
    e = e[:, order]
    pivot = np.argmax(np.abs(e), axis=0)
    sgn = np.sign(e[pivot, np.arange(e.shape[1])])
    sgn[sgn == 0] = 1.0
    return w, e * sgn[None, :]


def key_transform(mq: np.ndarray, sk: np.ndarray):
    """Theorem 1 closed form.

    A = M_q^{1/2} S_k M_q^{1/2} = E Lambda E^T;  R_K = M_q^{1/2} E;  R_K^{-T} = M_q^{-1/2} E.
    Returns (R_K, R_K^{-T}, lambda) with columns in decreasing-lambda order.
    """
    mq_half = sym_power(mq, 0.5)
    mq_ihalf = sym_power(mq, -0.5)
    lam, e = eig_descending(mq_half @ sk @ mq_half)
    return mq_half @ e, mq_ihalf @ e, lam


def causal_attention_outputs(q: np.ndarray, k: np.ndarray, v: np.ndarray, positions, scale: float):
    """o_i = softmax(q_i K_{0..i}^T * scale) V_{0..i} for the given query positions."""
    out = np.empty((len(positions), v.shape[1]))
    chunk = 256
    for a in range(0, len(positions), chunk):
        pos = np.asarray(positions[a:a + chunk])
        hi = pos.max() + 1
        z = (q[pos] @ k[:hi].T) * scale
        mask = np.arange(hi)[None, :] > pos[:, None]
        z[mask] = -np.inf
        z -= z.max(axis=1, keepdims=True)
        p = np.exp(z)
        p /= p.sum(axis=1, keepdims=True)
        out[a:a + len(pos)] = p @ v[:hi]
    return out


def output_second_moment(q_heads: np.ndarray, k: np.ndarray, v: np.ndarray,
                         stride: int, scale: float) -> np.ndarray:
    """M_o = V^T M_s V = sum_i o_i^T o_i (Corollary 1 proof), mean over heads and positions."""
    g, m, d = q_heads.shape
    positions = np.arange(stride - 1, m, stride)
    mo = np.zeros((d, d))
    for h in range(g):
        o = causal_attention_outputs(q_heads[h], k, v, positions, scale)
        mo += o.T @ o
    return mo / (g * len(positions))


def value_transform(mo: np.ndarray):
    """Corollary 1: R_V = eigenvectors of M_o (decreasing eigenvalues); orthogonal."""
    lam, e = eig_descending(mo)
    return e, lam


def value_grouping_order(v_cal: np.ndarray, r_v: np.ndarray) -> np.ndarray:
    """Columns of R_V ranked for the grouping: decreasing empirical variance of v R_V.

    Paper, Sec. "KV cache vector quantization" (the equalizing grouping deals
    coordinates sorted by decreasing variance) and Algorithm 2 (the same fold
    for the values).  The sort key for the values is the variance of the
    rotated calibration values (reading: for the keys it coincides with the
    eigenvalue order); ties keep the eigenvalue order.
    """
    var_v = (v_cal @ r_v).var(axis=0)
    return np.argsort(-var_v, kind="stable")


def equalizing_columns(d: int, g: int) -> np.ndarray:
    """Column position of each variance rank under the volume-equalizing partition.

    Paper, Theorem 2 discussion and Algorithm 2: after sorting by decreasing
    variance, rank r joins group r mod L (L = d / g); the partition is folded
    into the transform's column order.  Rank r goes to column (r mod L)*g + r//L.
    """
    L = d // g
    r = np.arange(d)
    return (r % L) * g + r // L


def fold_columns(mat_by_rank: np.ndarray, g: int) -> np.ndarray:
    """Reorder columns (given in rank order) into equalizing-group order."""
    d = mat_by_rank.shape[1]
    pos = equalizing_columns(d, g)
    out = np.empty_like(mat_by_rank)
    out[:, pos] = mat_by_rank
    return out


def calibrate_head(k_cal: np.ndarray, v_cal: np.ndarray, q_cal: np.ndarray, *,
                   group_dim: int = 4, codebook_size: int = 256, mo_stride: int = 16,
                   kmeans_iters: int = 25, seed=0, key_scale: bool = False):
    """Full per-(layer, KV head) calibration: Algorithms 2 and 3, Corollary 1.

    With key_scale the key codebooks are trained on the normalized coefficients
    r_j / rho_j, rho_j = ||r_j|| / sqrt(d) (Algorithm 2), for the key-scale format.

    Inputs: calibration keys (M, D), values (M, D) and the G sharing query heads'
    queries (G, M, D).  Returns a dict of stored parameters (t_k, t_k_inv_t,
    t_v, kbar in fp32; cb_k, cb_v in fp16 (L, k, g)) and fp64 diagnostics.
    """
    d = k_cal.shape[1]
    g = group_dim
    scale = 1.0 / np.sqrt(d)
    mq = query_second_moment(q_cal)
    kbar, sk = key_statistics(k_cal)
    r_k, r_k_inv_t, lam_k = key_transform(mq, sk)
    t_k = fold_columns(r_k, g)
    t_k_inv_t = fold_columns(r_k_inv_t, g)

    mo = output_second_moment(q_cal, k_cal, v_cal, mo_stride, scale)
    r_v, lam_v = value_transform(mo)
    t_v = fold_columns(r_v[:, value_grouping_order(v_cal, r_v)], g)

    stored = {
        "kbar": kbar.astype(np.float32),
        "t_k": t_k.astype(np.float32),
        "t_k_inv_t": t_k_inv_t.astype(np.float32),
        "t_v": t_v.astype(np.float32),
    }
    ss = seed if isinstance(seed, np.random.SeedSequence) else np.random.SeedSequence(seed)
    seed_k, seed_v = ss.spawn(2)
    r_cal = (k_cal - stored["kbar"].astype(np.float64)) @ stored["t_k"].astype(np.float64)
    s_cal_stored = v_cal @ stored["t_v"].astype(np.float64)
    if key_scale:
        r_cal = normalized_key_coefficients(r_cal)[0]
    stored["cb_k"] = train_codebooks(r_cal, g, codebook_size, seed_k, kmeans_iters)
    stored["cb_v"] = train_codebooks(s_cal_stored, g, codebook_size, seed_v, kmeans_iters)
    diag = {"m_q": mq, "s_k": sk, "m_o": mo, "lambda_k": lam_k, "lambda_v": lam_v,
            "r_k": r_k, "r_k_inv_t": r_k_inv_t, "r_v": r_v, "kbar64": kbar}
    return stored, diag


def stack_params(per_head):
    """Stack per-KV-head stored parameter dicts into [Hkv][...] arrays."""
    keys = ["kbar", "t_k", "t_k_inv_t", "t_v", "cb_k", "cb_v"]
    return {k: np.stack([p[k] for p in per_head]) for k in keys}
