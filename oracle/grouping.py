"""Oracle: Theorem 2 quantities (Zador high-resolution model, grouping, rate allocation).

Test infrastructure only (see ``oracle/__init__.py``).  Not used by the GPU
path; the grouping it motivates is folded into the transforms by
``calibration.fold_columns``.

Paper, Sec. "KV cache vector quantization": under the independent-Gaussian
high-resolution model, group l of g coefficients with b_l bits per entry has
distortion D_l = C_g 2^{-2 b_l} v_l^{1/g}, v_l = prod_{i in G_l} sigma_i^2 (its
volume).  Theorem 2 gives the optimal allocation
b*_l = b + (1/(2g)) log2(v_l / (prod_m v_m)^{1/L}) and the partition-independent
optimum D*(b) = C_g L 2^{-2b} (prod_i sigma_i^2)^{1/d}; at fixed rate b_l = b the
distortion is 2^{-2b} C_g sum_l v_l^{1/g} >= D*(b), with equality iff all volumes
are equal.
"""

from __future__ import annotations

import numpy as np


def sorted_partition(d: int, g: int):
    """Variance-sorted grouping: consecutive runs of g ranks."""
    return [list(range(ell * g, (ell + 1) * g)) for ell in range(d // g)]


def equalizing_partition(d: int, g: int):
    """Volume-equalizing grouping: rank i joins group i mod L."""
    L = d // g
    return [[i for i in range(d) if i % L == ell] for ell in range(L)]


def volumes(var: np.ndarray, partition) -> np.ndarray:
    return np.array([np.prod(np.asarray(var)[list(grp)]) for grp in partition])


def group_distortion(var, partition, rates, c_g: float = 1.0) -> np.ndarray:
    """D_l(b_l) = C_g 2^{-2 b_l} v_l^{1/g} per group."""
    g = len(partition[0])
    v = volumes(var, partition)
    return c_g * 2.0 ** (-2.0 * np.asarray(rates, dtype=np.float64)) * v ** (1.0 / g)


def optimal_rates(var, partition, b: float) -> np.ndarray:
    """Theorem 2 allocation b*_l."""
    g = len(partition[0])
    v = volumes(var, partition)
    L = len(partition)
    geo = np.exp(np.log(v).sum() / L)
    return b + np.log2(v / geo) / (2.0 * g)


def optimal_distortion(var, g: int, b: float, c_g: float = 1.0) -> float:
    """Theorem 2 optimum D*(b) = C_g L 2^{-2b} (prod sigma^2)^{1/d}."""
    var = np.asarray(var, dtype=np.float64)
    d = var.size
    return c_g * (d // g) * 2.0 ** (-2.0 * b) * np.exp(np.log(var).sum() / d)


def fixed_rate_distortion(var, partition, b: float, c_g: float = 1.0) -> float:
    """Distortion when every group gets the same rate b."""
    return float(group_distortion(var, partition, np.full(len(partition), b), c_g).sum())
