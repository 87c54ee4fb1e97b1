"""Oracle fp8 E4M3 snapping of the codebooks.

Test infrastructure only (see ``oracle/__init__.py``).

Paper, Sec. "Calibration" and the implementation table: each group's codebook
(per layer and KV head) is stored in fp16 and rounded to fp8 ahead of use.  The fp8
format is taken to be OCP E4M3 ("e4m3fn"): sign bit, 4 exponent bits with
bias 7, 3 mantissa bits, no infinities, the code with all exponent and
mantissa bits set is NaN; normals (-1)^s 2^(e-7) (1 + m/8), subnormals
(-1)^s 2^-6 (m/8); largest finite magnitude 448.  Readings: snapping rounds
the fp16 value to the nearest E4M3 value, ties to the even mantissa, and
saturates magnitudes above 448 to 448 (a codebook never holds a NaN).
"""

from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0
_MIN_NORMAL = 2.0 ** -6
_SUB_STEP = 2.0 ** -9


def e4m3_value(bits: np.ndarray) -> np.ndarray:
    """fp64 values of E4M3 codes (uint8); the NaN codes give NaN."""
    b = np.asarray(bits, dtype=np.int64)
    s = np.where(b & 0x80, -1.0, 1.0)
    e = (b >> 3) & 0xF
    m = (b & 7).astype(np.float64)
    v = np.where(e == 0, m / 8.0 * _MIN_NORMAL, np.ldexp(1.0 + m / 8.0, (e - 7).astype(np.int64)))
    v = np.where(((b & 0x7F) == 0x7F), np.nan, v)
    return s * v


def snap_e4m3(x: np.ndarray) -> np.ndarray:
    """Nearest E4M3 value of each element (ties to even, saturating at 448), as fp64."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    out = np.empty_like(a)
    sub = a < _MIN_NORMAL
    out[sub] = np.rint(a[sub] / _SUB_STEP) * _SUB_STEP          # rint: ties to even
    nrm = ~sub
    e = np.floor(np.log2(a[nrm]))
    step = np.ldexp(1.0, (e - 3).astype(np.int64))               # 8 values per binade
    out[nrm] = np.rint(a[nrm] / step) * step
    out = np.minimum(out, E4M3_MAX)
    return np.copysign(out, x)


def e4m3_bits(v: np.ndarray) -> np.ndarray:
    """E4M3 codes (uint8) of values that are exactly representable (e.g. snap_e4m3's)."""
    v = np.asarray(v, dtype=np.float64)
    s = np.signbit(v).astype(np.int64) << 7
    a = np.abs(v)
    bits = np.zeros(a.shape, dtype=np.int64)
    sub = (a < _MIN_NORMAL) & (a > 0)
    bits[sub] = np.rint(a[sub] / _SUB_STEP).astype(np.int64)
    nrm = a >= _MIN_NORMAL
    e = np.floor(np.log2(a[nrm])).astype(np.int64)
    m = np.rint((a[nrm] / np.ldexp(1.0, e) - 1.0) * 8.0).astype(np.int64)
    bits[nrm] = ((e + 7) << 3) | m
    out = (bits | s).astype(np.uint8)
    assert np.all(e4m3_value(out) == v), "value not representable in E4M3"
    return out


def snap_codebooks(cb: np.ndarray) -> np.ndarray:
    """fp16 codebooks [..., 256, 4] snapped to E4M3, returned as fp16 (every E4M3 value is exact in fp16)."""
    return snap_e4m3(np.asarray(cb, dtype=np.float16).astype(np.float64)).astype(np.float16)
