"""Test-side plumbing: code pools on the host, parity comparisons."""

from __future__ import annotations

import numpy as np

TOL = 2e-3          # max-abs error relative to the output row's L2 norm
NEAR_TIE = 1e-6     # squared-distance gap under which a code mismatch is a near-tie

# Parity report of the session: one entry per comparison, written by
# conftest.py at the end of the session (codes compared, mismatches, near-ties,
# near-tie mismatches; output rows compared and the worst row error).
REPORT = []
CURRENT_TEST = {"id": ""}


def _record(kind, what, **fields):
    REPORT.append({"test": CURRENT_TEST["id"], "kind": kind, "what": what, **fields})


def pool_offsets(b, kv, t, *, hkv, groups, block_size, blocks_per_seq, table=None):
    """Byte offsets of the code rows of tokens t (array) of sequence b, KV head kv."""
    t = np.asarray(t)
    blk = t // block_size
    row = t % block_size
    logical = b * blocks_per_seq + blk
    phys = table.reshape(-1)[logical] if table is not None else logical
    return ((phys.astype(np.int64) * hkv + kv) * block_size + row) * groups


def write_rows(pool: np.ndarray, codes: np.ndarray, b, kv, start, **lay):
    """Write code rows (n, L) of (b, kv) at positions start.. into a flat host pool."""
    n, L = codes.shape
    off = pool_offsets(b, kv, np.arange(start, start + n), groups=L, **lay)
    idx = off[:, None] + np.arange(L)[None, :]
    pool[idx] = codes


def read_rows(pool: np.ndarray, b, kv, start, n, *, groups, **lay):
    off = pool_offsets(b, kv, np.arange(start, start + n), groups=groups, **lay)
    return pool[off[:, None] + np.arange(groups)[None, :]]


def row_errors(gpu: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """max_i |gpu - ref| / ||ref||_2 per output row (last axis)."""
    num = np.abs(gpu - ref).max(axis=-1)
    den = np.linalg.norm(ref, axis=-1)
    return np.where(den > 0, num / np.maximum(den, 1e-300), num)


def assert_outputs_close(gpu, ref, tol=TOL, what=""):
    err = row_errors(np.asarray(gpu, dtype=np.float64), np.asarray(ref, dtype=np.float64))
    worst = float(err.max()) if err.size else 0.0
    print(f"[parity] {what} rows={err.size} worst_rel_err={worst:.3e} tol={tol}", flush=True)
    _record("output", what, rows=int(err.size), worst_rel_err=worst, tol=tol, ok=bool(worst <= tol))
    assert worst <= tol, f"{what}: worst relative row error {worst:.3e} > {tol}"
    return worst


def compare_codes(gpu_codes, ref_codes, ref_gap, what=""):
    """Codes must match bit-exactly except where the oracle's top-2 gap is a near-tie."""
    gpu_codes = np.asarray(gpu_codes)
    mism = gpu_codes != ref_codes
    near = ref_gap < NEAR_TIE
    bad = mism & ~near
    n_near = int(near.sum())
    print(f"[parity] {what} codes={gpu_codes.size} mismatches={int(mism.sum())} "
          f"near_ties={n_near} near_tie_mismatches={int((mism & near).sum())}", flush=True)
    _record("codes", what, codes=int(gpu_codes.size), mismatches=int(mism.sum()), near_ties=n_near,
            near_tie_mismatches=int((mism & near).sum()), ok=not bool(bad.any()))
    assert not bad.any(), f"{what}: {int(bad.sum())} code mismatches outside near-ties"
    return int(mism.sum()), n_near
