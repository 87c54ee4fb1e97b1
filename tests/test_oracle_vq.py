"""Pins for the oracle's encoder, Lloyd training and lookup decoder."""

import itertools

import numpy as np
import pytest
from scipy.spatial import cKDTree

from oracle import vq


def test_nearest_matches_kdtree():
    """Exhaustive search agrees with an independent nearest-neighbour library."""
    rng = np.random.default_rng(0)
    u = rng.standard_normal((5000, 4)) * 2
    cb = rng.standard_normal((256, 4)) * 2
    codes, best, second = vq.nearest_codeword(u, cb)
    dist, idx = cKDTree(cb).query(u, k=2)
    assert np.array_equal(codes, idx[:, 0])
    assert np.allclose(best, dist[:, 0] ** 2, rtol=1e-12)
    assert np.allclose(second, dist[:, 1] ** 2, rtol=1e-12)


def test_grid_codebook_is_coordinate_rounding():
    """Codewords on the grid {0,1,2,3}^4: the nearest one rounds each coordinate and clips."""
    grid = np.array(list(itertools.product(range(4), repeat=4)), dtype=np.float64)   # 256 points
    rng = np.random.default_rng(1)
    u = rng.uniform(-1.2, 4.2, (3000, 4))
    u = u[np.all(np.abs(u - np.floor(u) - 0.5) > 0.01, axis=1)]      # no rounding ties
    codes, _, _ = vq.nearest_codeword(u, grid)
    expect = np.clip(np.floor(u + 0.5), 0, 3)
    assert np.array_equal(grid[codes], expect)


def test_ties_take_lowest_index():
    cb = np.array([[1.0, 0, 0, 0], [0, 1.0, 0, 0], [1.0, 0, 0, 0], [0, 0, 0, 0]])
    u = np.array([[1.0, 0, 0, 0], [0.5, 0.5, 0, 0]])
    codes, best, second = vq.nearest_codeword(u, cb)
    assert list(codes) == [0, 0]         # duplicate codeword 2 loses to 0; equidistant 0 vs 1 -> 0
    assert second[0] == best[0] and second[1] == best[1]


def test_lloyd_monotone_and_deterministic():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((4000, 4)) * np.array([3.0, 1.0, 0.5, 0.2])
    c1, hist = vq.lloyd(x, 64, seed=7, max_iter=25, return_history=True)
    c2 = vq.lloyd(x, 64, seed=7, max_iter=25)
    assert np.array_equal(c1, c2)
    assert all(b <= a * (1 + 1e-12) for a, b in zip(hist, hist[1:]))
    assert len(hist) <= 26


def test_lloyd_lossless_on_few_distinct_points():
    """At most k distinct training points: Lloyd reaches zero distortion (exact codebook)."""
    rng = np.random.default_rng(3)
    atoms = np.round(rng.standard_normal((200, 4)) * 8) / 8
    x = atoms[rng.integers(0, 200, 6000)]
    cent, hist = vq.lloyd(x, 256, seed=1, return_history=True)
    _, best, _ = vq.nearest_codeword(x, cent)
    assert hist[-1] == 0.0 and best.max() == 0.0


def test_lloyd_matches_sklearn_from_same_start():
    """Same initial centroids, no empty clusters: identical to scikit-learn's Lloyd."""
    from sklearn.cluster import KMeans
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3000, 4)) * np.array([2.0, 1.0, 0.7, 0.4])
    k = 16
    init_idx = np.random.default_rng(9).choice(3000, size=k, replace=False)
    ours = vq.lloyd(x, k, seed=9, max_iter=25)
    km = KMeans(n_clusters=k, init=x[init_idx], n_init=1, max_iter=25, tol=0.0,
                algorithm="lloyd").fit(x)
    order = np.lexsort(ours.T[::-1])
    order2 = np.lexsort(km.cluster_centers_.T[::-1])
    assert np.allclose(ours[order], km.cluster_centers_[order2], atol=1e-10)


def test_encode_and_lookup_roundtrip():
    rng = np.random.default_rng(5)
    books = rng.standard_normal((8, 256, 4)).astype(np.float16)
    codes_true = rng.integers(0, 256, (100, 8)).astype(np.uint8)
    x = vq.lookup(codes_true, books)                       # points exactly on codewords
    codes, gap = vq.encode(x, books)
    dup = np.zeros_like(codes, dtype=bool)
    for ell in range(8):
        u, inv, cnt = np.unique(books[ell].astype(np.float64), axis=0, return_inverse=True,
                                return_counts=True)
        dup[:, ell] = cnt[inv.ravel()[codes_true[:, ell]]] > 1
    assert np.array_equal(codes[~dup], codes_true[~dup])
    assert np.array_equal(vq.lookup(codes, books), x)
    assert np.all(gap >= 0)


# ---- Lloyd's start and its refill of empty clusters (Sec. "Calibration"; Algorithm 3)

def _two_far_points():
    """1000 copies of the origin and two outliers, at squared distances 100 and 400."""
    x = np.zeros((1002, 4))
    x[1000, 0] = 10.0   # F1
    x[1001, 0] = 20.0   # F2
    return x


def check_refill(lloyd_fn):
    """Three clusters started on copies of the origin: two are empty after the
    first assignment (equal centroids, ties to the lowest index) and must be
    refilled from the worst-fit points, the farthest first.  Seed 3 starts on
    three origin copies (distortion 100 + 400 at the first assignment).
    Afterwards cluster 0 sits at the origin, cluster 1 at the farther outlier,
    cluster 2 at the nearer one, and the training distortion is zero."""
    x = _two_far_points()
    cent, hist = lloyd_fn(x, 3, seed=3, max_iter=25, return_history=True)
    assert hist[0] == 500.0, "the start was not three copies of the origin"
    return (np.array_equal(cent[0], x[0]) and np.array_equal(cent[1], x[1001])
            and np.array_equal(cent[2], x[1000]) and hist[-1] == 0.0)


def test_lloyd_refills_empty_clusters_from_the_worst_fit_points():
    assert check_refill(vq.lloyd)


@pytest.mark.parametrize("mistake", ["nearest", "increasing"])
def test_lloyd_refill_pin_catches_planted_mistakes(monkeypatch, mistake):
    """The refill pin fails when the refill takes the best-fit points, or the
    worst-fit points in increasing order of their distance."""
    fn = {"nearest": lambda best, n: np.argsort(best, kind="stable")[:n],
          "increasing": lambda best, n: np.argsort(-best, kind="stable")[:n][::-1]}[mistake]
    monkeypatch.setattr(vq, "reseed_indices", fn)
    assert not check_refill(vq.lloyd)


def test_lloyd_starts_on_distinct_training_points():
    """k distinct points and n = k: a start on k distinct indices is already the
    lossless codebook (zero distortion at the first assignment)."""
    rng = np.random.default_rng(12)
    x = rng.standard_normal((256, 4))
    _, hist = vq.lloyd(x, 256, seed=5, return_history=True)
    assert hist[0] == 0.0 and len(hist) == 2      # nothing moves: stop after the second assignment


def test_lloyd_start_pin_catches_draws_with_replacement(monkeypatch):
    rng = np.random.default_rng(12)
    x = rng.standard_normal((256, 4))
    monkeypatch.setattr(vq, "initial_indices", lambda r, n, k: r.choice(n, size=k, replace=True))
    _, hist = vq.lloyd(x, 256, seed=5, return_history=True)
    assert hist[0] > 0.0
