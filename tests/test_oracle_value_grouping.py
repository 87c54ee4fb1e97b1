"""Pin of the value-side grouping (Sec. "KV cache vector quantization": the
equalizing grouping deals coordinates sorted by decreasing variance to the
groups in turn; Algorithm 2: the grouping is folded into the transform's
columns; for the values the sort key is the variance of the rotated
calibration values).

A D = 16 value distribution is built so that the three plausible sort keys
disagree: a large mean along one direction a with almost no spread along it
(so a is the top eigenvector of M_o = E[o o^T] but has the smallest variance),
and distinct spreads sigma_i along the other directions of a random basis.
With L = 4 groups, column 4l + j of t_v must carry the coordinate of variance
rank l + 4j (rank 0 = largest).
"""

import numpy as np
import pytest

from oracle import calibration

D, G, M = 16, 2, 4096
# rank r -> column (r mod L) * 4 + r // L, written out for L = 4
EXPECTED_COLUMN_OF_RANK = [0, 4, 8, 12, 1, 5, 9, 13, 2, 6, 10, 14, 3, 7, 11, 15]


def _data():
    rng = np.random.default_rng(2024)
    basis, _ = np.linalg.qr(rng.standard_normal((D, D)))
    a = basis[:, 0]
    sig = np.concatenate([[0.02], 3.0 * 0.8 ** np.arange(1, D)])
    v = 5.0 * a[None, :] + (rng.standard_normal((M, D)) * sig[None, :]) @ basis.T
    k = rng.standard_normal((M, D))
    q = rng.standard_normal((G, M, D))
    return k, v, q, a


def _calibrate(k, v, q):
    stored, diag = calibration.calibrate_head(k, v, q, mo_stride=16, kmeans_iters=2, seed=[7])
    return stored, diag


def grouping_ok(stored, v):
    s = v @ stored["t_v"].astype(np.float64)
    ranked = np.argsort(-s.var(axis=0), kind="stable")     # columns by decreasing variance
    return list(ranked) == EXPECTED_COLUMN_OF_RANK


@pytest.fixture(scope="module")
def data():
    return _data()


def test_value_columns_carry_the_dealt_variance_ranks(data):
    k, v, q, a = data
    stored, diag = _calibrate(k, v, q)
    assert grouping_ok(stored, v)
    # the construction works as intended: the top eigenvector of M_o is the
    # mean direction, whose variance is the smallest, so it sits in the last
    # column (rank 15)
    top = diag["r_v"][:, 0]
    assert abs(top @ a) > 0.999
    last = stored["t_v"][:, EXPECTED_COLUMN_OF_RANK[15]].astype(np.float64)
    assert abs(last @ a) > 0.999


@pytest.mark.parametrize("mistake", ["ascending", "eigenvalue_order", "raw_coordinates"])
def test_value_grouping_pin_catches_planted_mistakes(data, monkeypatch, mistake):
    """An ascending sort, the eigenvalue order of M_o, or the variances of the
    unrotated values each break the dealing."""
    k, v, q, _ = data
    wrong = {
        "ascending": lambda vc, rv: np.argsort((vc @ rv).var(axis=0), kind="stable"),
        "eigenvalue_order": lambda vc, rv: np.arange(rv.shape[1]),
        "raw_coordinates": lambda vc, rv: np.argsort(-vc.var(axis=0), kind="stable"),
    }[mistake]
    monkeypatch.setattr(calibration, "value_grouping_order", wrong)
    stored, _ = _calibrate(k, v, q)
    assert not grouping_ok(stored, v)
