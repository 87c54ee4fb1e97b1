"""Oracle vector quantizer: exhaustive encoder, Lloyd codebook training, lookup decoder.

Test infrastructure only (see ``oracle/__init__.py``).
"""

from __future__ import annotations

import ctypes

import numpy as np

from .build import ensure_built

_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(ensure_built())
        fn = lib.oracle_nearest_codeword
        fn.restype = None
        fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                       ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        _lib = lib
    return _lib


def nearest_codeword(u: np.ndarray, codebook: np.ndarray):
    """Exhaustive nearest codeword of each row of ``u`` (n, g) in ``codebook`` (k, g).

    Paper, Sec. "Transform coding" (quantization): the encoder returns the
    index of the nearest codeword; Sec. "Calibration": exact nearest-neighbour
    search in the Euclidean metric.  Ties go to the lowest index.

    Returns (codes int32 (n,), best (n,), second (n,)) with squared distances in fp64.
    """
    u = np.ascontiguousarray(u, dtype=np.float64)
    n, g = u.shape
    cb_t = np.ascontiguousarray(np.asarray(codebook, dtype=np.float64).T)
    k = cb_t.shape[1]
    codes = np.empty(n, dtype=np.int32)
    best = np.empty(n)
    second = np.empty(n)
    if n:
        _load().oracle_nearest_codeword(u.ctypes.data, n, g, cb_t.ctypes.data, k,
                                        codes.ctypes.data, best.ctypes.data, second.ctypes.data)
    return codes, best, second


def initial_indices(rng: np.random.Generator, n: int, k: int) -> np.ndarray:
    """Training points that start Lloyd: k distinct indices, uniformly without replacement."""
    return rng.choice(n, size=k, replace=False)


def reseed_indices(best: np.ndarray, n_empty: int) -> np.ndarray:
    """Training points that refill empty clusters: the worst-fit points first.

    ``best`` holds each point's squared distance to the centroid it was
    assigned to; the n_empty points with the largest such distance are taken
    in decreasing order of it (equal distances in index order), so the i-th
    empty cluster gets the i-th worst-fit point (Sec. "Calibration").
    """
    return np.argsort(-best, kind="stable")[:n_empty]


def lloyd(points: np.ndarray, k: int, seed, max_iter: int = 25, return_history: bool = False):
    """k-means (Lloyd) codebook for one group, in fp64.

    Paper, Algorithm 3 and Sec. "Calibration": k-means from a random start,
    no more than 25 iterations, and every iteration refills empty clusters
    from the worst-fit training points.

    Readings where the paper is silent:
      * initialisation: k distinct training points drawn uniformly without
        replacement from ``np.random.default_rng(seed)``;
      * each iteration assigns every point to its nearest centroid (lowest index
        on ties), stops if no assignment changed, then moves every non-empty
        centroid to the mean of its points;
      * empty clusters, in index order, take the training points with the
        largest distance to their assigned centroid, in decreasing order of
        that distance (each point used once).

    Returns the fp64 centroids (k, g); with ``return_history`` also the
    training distortion (sum of squared distances) at every assignment step.
    """
    x = np.ascontiguousarray(points, dtype=np.float64)
    n, g = x.shape
    rng = np.random.default_rng(seed)
    if n < k:
        raise ValueError("need at least k training points")
    cent = x[initial_indices(rng, n, k)].copy()
    prev = None
    history = []
    for _ in range(max_iter):
        assign, best, _ = nearest_codeword(x, cent)
        history.append(float(best.sum()))
        if prev is not None and np.array_equal(assign, prev):
            break
        prev = assign
        counts = np.bincount(assign, minlength=k)
        sums = np.zeros((k, g))
        np.add.at(sums, assign, x)
        nonempty = counts > 0
        cent[nonempty] = sums[nonempty] / counts[nonempty, None]
        empty = np.flatnonzero(~nonempty)
        if empty.size:
            cent[empty] = x[reseed_indices(best, empty.size)]
    else:
        assign, best, _ = nearest_codeword(x, cent)
        history.append(float(best.sum()))
    if return_history:
        return cent, history
    return cent


def to_fp16(cent: np.ndarray) -> np.ndarray:
    """Store a codebook in fp16 (round to nearest even), as the paper stores codebooks."""
    return np.asarray(cent, dtype=np.float64).astype(np.float16)


def train_codebooks(coeffs: np.ndarray, group_dim: int, k: int, seed, max_iter: int = 25):
    """One k-entry codebook per group of ``group_dim`` consecutive coefficients.

    Paper, Algorithm 3: one codebook per group, equal size for every group,
    trained on the grouped transform coefficients.  Returns fp16 (L, k, g).
    """
    m, d = coeffs.shape
    L = d // group_dim
    ss = seed if isinstance(seed, np.random.SeedSequence) else np.random.SeedSequence(seed)
    children = ss.spawn(L)
    books = []
    for ell in range(L):
        pts = coeffs[:, ell * group_dim:(ell + 1) * group_dim]
        books.append(to_fp16(lloyd(pts, k, children[ell], max_iter)))
    return np.stack(books)


def encode(coeffs: np.ndarray, codebooks: np.ndarray):
    """Codes of transform coefficients (n, D) against per-group codebooks (L, k, g).

    Returns (codes uint8 (n, L), gap (n, L)) where gap = second-best minus best
    squared distance (the near-tie margin).
    """
    n, d = coeffs.shape
    L, k, g = codebooks.shape
    codes = np.empty((n, L), dtype=np.uint8)
    gap = np.empty((n, L))
    cb = codebooks.astype(np.float64)
    for ell in range(L):
        c, b1, b2 = nearest_codeword(coeffs[:, ell * g:(ell + 1) * g], cb[ell])
        codes[:, ell] = c
        gap[:, ell] = b2 - b1
    return codes, gap


def lookup(codes: np.ndarray, codebooks: np.ndarray) -> np.ndarray:
    """Decoder: concatenate, per group, the codeword each index selects (n, L*g) fp64.

    Paper, Sec. "Decoding kernel and read path": the stored 8-bit index of each
    group selects a g-dimensional centroid from that group's codebook.
    """
    codes = np.asarray(codes)
    L, k, g = codebooks.shape
    cb = codebooks.astype(np.float64)
    parts = [cb[ell][codes[:, ell].astype(np.int64)] for ell in range(L)]
    return np.concatenate(parts, axis=1)
