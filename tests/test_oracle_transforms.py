"""Pins for the oracle's calibration transforms (Theorem 1, Proposition 1, Corollary 1).

Each check compares the oracle against something other than itself: brute-force
numeric minimisation of the paper's objectives, library eigen/SVD routines,
explicitly formed matrices, or identities the paper proves.
"""

import numpy as np
import pytest
from scipy.optimize import minimize

from oracle import calibration as cal


def _spd(rng, d, spread=10.0):
    u, _ = np.linalg.qr(rng.standard_normal((d, d)))
    w = np.exp(rng.uniform(0, np.log(spread), d))
    return (u * w) @ u.T


def _keys(rng, m, d):
    a = rng.standard_normal((d, d)) * np.linspace(2.0, 0.3, d)[None, :]
    return rng.standard_normal((m, d)) @ a + rng.standard_normal(d)


def test_parseval_identity_d4():
    """Prop. 1: ||r - r_hat||^2 = ||k - k_hat||^2_{M_q} for any r, r_hat, k = r R_K^{-1}."""
    rng = np.random.default_rng(1)
    d = 4
    mq = _spd(rng, d)
    k = _keys(rng, 200, d)
    _, sk = cal.key_statistics(k)
    r_k, _, _ = cal.key_transform(mq, sk)
    inv = np.linalg.inv(r_k)
    for _ in range(20):
        r = rng.standard_normal(d) * 3
        rh = rng.standard_normal(d) * 3
        e = r @ inv - rh @ inv
        assert np.isclose(np.sum((r - rh) ** 2), e @ mq @ e, rtol=1e-11, atol=1e-12)


def test_parseval_attention_products_d4():
    """Attention-product error equals transform-domain MSE (summed Prop. 1 / Eq. qmse + GQA).

    sum_h ||Q_h K^T - Q_h K_hat^T||_F^2 = G*M * sum_j ||r_j - r_hat_j||^2 when
    M_q is the mean second moment over G heads and M queries each.
    """
    rng = np.random.default_rng(2)
    d, m, g = 4, 300, 3
    qh = np.stack([rng.standard_normal((m, d)) @ _spd(rng, d, 5.0) for _ in range(g)])
    k = _keys(rng, 257, d)
    mq = cal.query_second_moment(qh)
    kbar, sk = cal.key_statistics(k)
    r_k, r_k_inv_t, _ = cal.key_transform(mq, sk)
    r = (k - kbar) @ r_k
    r_hat = np.round(r * 2.0) / 2.0            # any quantizer works: a coarse grid
    k_hat = r_hat @ r_k_inv_t.T + kbar         # R_K^{-1} = (R_K^{-T})^T
    lhs = sum(np.sum((qh[h] @ k.T - qh[h] @ k_hat.T) ** 2) for h in range(g))
    rhs = g * m * np.sum((r - r_hat) ** 2)
    assert np.isclose(lhs, rhs, rtol=1e-10)


def test_key_transform_invariants():
    rng = np.random.default_rng(3)
    d = 16
    mq = _spd(rng, d, 50.0)
    k = _keys(rng, 1000, d)
    _, sk = cal.key_statistics(k)
    r_k, r_k_inv_t, lam = cal.key_transform(mq, sk)
    assert np.allclose(r_k @ r_k.T, mq, rtol=0, atol=1e-11 * np.abs(mq).max())     # R R^T = M_q
    assert np.allclose(r_k_inv_t, np.linalg.inv(r_k).T, atol=1e-10)                 # R^{-T}
    cov = r_k.T @ sk @ r_k                                                           # decorrelated,
    assert np.allclose(cov, np.diag(lam), atol=1e-10 * lam.max())                    # variances = lambda
    assert np.all(np.diff(lam) <= 0)
    # the grouping fold is a column permutation: invariants survive it
    t = cal.fold_columns(r_k, 4)
    assert np.allclose(t @ t.T, mq, atol=1e-11 * np.abs(mq).max())


def test_isotropic_query_reduces_to_pca():
    """Remark after Theorem 1: M_q proportional to I gives mean-centred PCA of the keys."""
    rng = np.random.default_rng(4)
    d = 8
    k = _keys(rng, 500, d)
    kbar, sk = cal.key_statistics(k)
    c = 2.5
    r_k, _, lam = cal.key_transform(c * np.eye(d), sk)
    _, s, vt = np.linalg.svd(k - k.mean(axis=0), full_matrices=False)
    # columns equal sqrt(c) times the principal directions, up to sign
    for i in range(d):
        col = r_k[:, i] / np.sqrt(c)
        assert np.isclose(abs(col @ vt[i]), 1.0, atol=1e-9)
    assert np.allclose(lam, c * s ** 2 / k.shape[0], rtol=1e-9)


def _weighted_pinv(r, mq_inv):
    return np.linalg.solve(r.T @ mq_inv @ r, r.T @ mq_inv)


def _thm1_objective(r_flat, kc, mq, mq_inv, p):
    r = r_flat.reshape(kc.shape[1], p)
    proj = r @ _weighted_pinv(r, mq_inv)
    e = kc - kc @ proj
    return np.einsum("ij,jk,ik->", e, mq, e)


@pytest.mark.parametrize("p", [1, 2, 3])
def test_thm1_matches_brute_force_d4(p):
    """Theorem 1 closed form attains the minimum of its objective (found numerically).

    The optimum value is sum_{i>p} lambda_i(A) (proof of Theorem 1) and the
    M_q-weighted projector R R^dagger agrees with the brute-force minimiser's.
    """
    rng = np.random.default_rng(10 + p)
    d = 4
    mq = _spd(rng, d, 8.0)
    k = _keys(rng, 400, d)
    kbar, sk = cal.key_statistics(k)
    kc = k - kbar
    mq_inv = np.linalg.inv(mq)
    r_k, _, lam = cal.key_transform(mq, sk)
    closed = _thm1_objective(r_k[:, :p].ravel(), kc, mq, mq_inv, p)
    best = None
    for _ in range(12):
        x0 = rng.standard_normal(d * p)
        res = minimize(_thm1_objective, x0, args=(kc, mq, mq_inv, p), method="BFGS",
                       options={"gtol": 1e-10, "maxiter": 5000})
        if best is None or res.fun < best.fun:
            best = res
    m = k.shape[0]
    assert np.isclose(closed, m * lam[p:].sum(), rtol=1e-9)
    assert np.isclose(best.fun, closed, rtol=1e-6)
    r_bf = best.x.reshape(d, p)
    proj_bf = r_bf @ _weighted_pinv(r_bf, mq_inv)
    proj_cf = r_k[:, :p] @ _weighted_pinv(r_k[:, :p], mq_inv)
    assert np.allclose(proj_bf, proj_cf, atol=1e-4)


def _causal_scores(q, k, scale):
    m = q.shape[0]
    z = (q @ k.T) * scale
    z[np.triu_indices(m, 1)] = -np.inf
    z -= z.max(axis=1, keepdims=True)
    s = np.exp(z)
    return s / s.sum(axis=1, keepdims=True)


def test_output_second_moment_equals_vt_ms_v():
    """Corollary 1 proof: M_o = V^T M_s V with M_s = S^T S, equal to sum_i o_i^T o_i."""
    rng = np.random.default_rng(5)
    d, m, g = 4, 37, 2
    qh = rng.standard_normal((g, m, d))
    k = rng.standard_normal((m, d))
    v = rng.standard_normal((m, d))
    scale = 0.5
    mo = cal.output_second_moment(qh, k, v, stride=1, scale=scale)
    explicit = np.zeros((d, d))
    for h in range(g):
        s = _causal_scores(qh[h], k, scale)
        explicit += v.T @ (s.T @ s) @ v
    assert np.allclose(mo, explicit / (g * m), atol=1e-13)


def _cor1_objective(d_flat, o, alphas_v, p, d):
    dv = d_flat.reshape(p, d)
    proj = dv.T @ np.linalg.solve(dv @ dv.T, dv)
    return np.sum((o - o @ proj) ** 2)


@pytest.mark.parametrize("p", [1, 2, 3])
def test_cor1_matches_brute_force_d4(p):
    """Corollary 1: R_V = top-p eigenvectors of M_o minimise ||S V - S V P||_F^2."""
    rng = np.random.default_rng(20 + p)
    d, m = 4, 60
    q = rng.standard_normal((m, d)) * 1.5
    k = rng.standard_normal((m, d))
    v = rng.standard_normal((m, d)) @ np.diag([3.0, 1.5, 0.8, 0.3])
    s = _causal_scores(q, k, 0.5)
    o = s @ v                                   # calibration outputs o_i
    mo = cal.output_second_moment(q[None], k, v, stride=1, scale=0.5) * m
    r_v, lam = cal.value_transform(mo)
    assert np.allclose(r_v.T @ r_v, np.eye(d), atol=1e-12)            # orthogonal
    closed = _cor1_objective(r_v[:, :p].T.ravel(), o, None, p, d)
    assert np.isclose(closed, lam[p:].sum(), rtol=1e-9)
    best = min((minimize(_cor1_objective, rng.standard_normal(p * d), args=(o, None, p, d),
                         method="BFGS", options={"gtol": 1e-11}) for _ in range(10)),
               key=lambda r: r.fun)
    assert np.isclose(best.fun, closed, rtol=1e-6)


def test_gqa_query_statistic():
    """Appendix GQA: sum_h ||Q_h (K - K_hat)^T||^2 = sum_j e_j (sum_h M_q^(h)) e_j^T."""
    rng = np.random.default_rng(6)
    d, m, g = 6, 50, 4
    qh = rng.standard_normal((g, m, d))
    e = rng.standard_normal((30, d))
    lhs = sum(np.sum((qh[h] @ e.T) ** 2) for h in range(g))
    mq = cal.query_second_moment(qh) * (g * m)
    rhs = np.einsum("ij,jk,ik->", e, mq, e)
    assert np.isclose(lhs, rhs, rtol=1e-11)


def test_eigen_floor():
    """M_q^{+-1/2} with eigenvalues floored at 1e-30 (calibration appendix)."""
    a = np.diag([4.0, 1.0, 0.0])
    h = cal.sym_power(a, 0.5)
    ih = cal.sym_power(a, -0.5)
    assert np.allclose(np.diag(h), [2.0, 1.0, 1e-15])
    assert np.allclose(np.diag(ih), [0.5, 1.0, 1e15])
