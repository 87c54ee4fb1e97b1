"""Pins for the grouping fold and the Theorem 2 closed forms."""

import os

import numpy as np
from scipy.optimize import minimize

from oracle import calibration as cal
from oracle import grouping as grp

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_toy():
    rules = {}
    with open(os.path.join(GOLDEN, "grouping_toy_d12_g4.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                name, *ids = line.split()
                rules[name] = [int(x) for x in ids]
    return rules


def test_toy_example_partitions():
    """The paper's d=12, g=4, L=3 toy figure: sorted and equalizing group memberships."""
    toy = _read_toy()
    for rule, parts in (("sorted", grp.sorted_partition(12, 4)),
                        ("equalizing", grp.equalizing_partition(12, 4))):
        member = [None] * 12
        for ell, members in enumerate(parts):
            for i in members:
                member[i] = ell
        assert member == toy[rule]


def test_fold_places_ranks_by_equalizing_groups():
    """The folded transform's group l (columns 4l..4l+3) holds exactly the ranks of group l."""
    toy = _read_toy()["equalizing"]
    pos = cal.equalizing_columns(12, 4)
    for rank in range(12):
        assert pos[rank] // 4 == toy[rank]
    # inside a group the ranks keep decreasing variance
    m = np.tile(np.arange(12.0), (2, 1))
    f = cal.fold_columns(m, 4)
    for ell in range(3):
        assert list(f[0, 4 * ell:4 * ell + 4]) == [ell, ell + 3, ell + 6, ell + 9]


def test_theorem2_allocation_is_the_constrained_minimum():
    """b*_l minimises sum_l D_l(b_l) subject to sum_l b_l = L b (numeric check)."""
    rng = np.random.default_rng(0)
    var = np.sort(rng.uniform(0.05, 9.0, 16))[::-1]
    b = 2.0
    for part in (grp.sorted_partition(16, 4), grp.equalizing_partition(16, 4)):
        L = len(part)
        cons = {"type": "eq", "fun": lambda x: x.sum() - L * b}
        res = minimize(lambda x: grp.group_distortion(var, part, x).sum(), np.full(L, b),
                       constraints=[cons], method="SLSQP", options={"ftol": 1e-15, "maxiter": 500})
        bstar = grp.optimal_rates(var, part, b)
        assert np.isclose(bstar.sum(), L * b)
        assert np.allclose(res.x, bstar, atol=1e-4)
        dl = grp.group_distortion(var, part, bstar)
        assert np.allclose(dl, dl[0], rtol=1e-10)                       # equal per-group distortion
        assert np.isclose(dl.sum(), grp.optimal_distortion(var, 4, b), rtol=1e-10)


def test_fixed_rate_gap_and_equal_volume_case():
    rng = np.random.default_rng(1)
    var = np.sort(rng.uniform(0.05, 9.0, 16))[::-1]
    b = 2.0
    dstar = grp.optimal_distortion(var, 4, b)
    d_sorted = grp.fixed_rate_distortion(var, grp.sorted_partition(16, 4), b)
    d_equal = grp.fixed_rate_distortion(var, grp.equalizing_partition(16, 4), b)
    assert d_sorted >= dstar and d_equal >= dstar              # AM-GM
    assert d_equal <= d_sorted                                   # dealing narrows the volume spread
    # equal volumes reach D*(b) exactly
    base = np.array([4.0, 2.0, 1.0, 0.5])
    var_eq = np.concatenate([base, base[::-1], base, base[[1, 0, 3, 2]]])
    part = grp.sorted_partition(16, 4)
    assert np.isclose(grp.fixed_rate_distortion(var_eq, part, b),
                      grp.optimal_distortion(var_eq, 4, b), rtol=1e-12)
