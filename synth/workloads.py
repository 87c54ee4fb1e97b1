"""Workload definitions and seeded generators.

Every array here is a pure function of (workload, layer, kv head, role, index),
drawn from NumPy's PCG64 seeded by ``SeedSequence([config_id, layer, kv_head,
role, index])``.  Floating-point tensors are rounded once to the workload's
storage dtype (fp32 or bf16) and returned as float64 arrays holding exactly the
stored values, so whoever consumes them (CPU oracle or GPU) sees identical
inputs.

The statistical model stands in for post-RoPE keys, values and queries of the
paper's models (Qwen3-8B: 32 query / 8 KV heads, head_dim 128; GPT-OSS-20B:
64 / 8 heads, head_dim 64, 128-token sliding windows and learned sinks), whose
activations are not available here:

* keys ~ N(0, U_k diag(lam_k) U_k^T), values ~ N(0, U_v diag(lam_v) U_v^T) with
  Haar-random orthogonal U_k, U_v per (layer, KV head);
* queries ~ N(0, U_q diag(lam_q) U_q^T), U_q = U_k (aligned) unless the workload
  asks for an independent basis;
* spectra lam_i proportional to i^-alpha, scaled to trace D (unit mean
  variance per coordinate).
"""

from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "get_workload", "ROLE",
    "rng_for", "haar_orthogonal", "power_spectrum", "round_to_bf16", "to_storage",
    "head_bases", "calibration_set", "cache_tokens", "decode_queries",
    "sink_logits", "random_codes", "random_key_scales", "shuffled_block_table",
    "uniform_seq_lens", "bench_params", "device_cache_tokens",
]

ROLE = {
    "basis_k": 0, "basis_v": 1, "basis_q": 2,
    "calib_k": 3, "calib_v": 4, "calib_q": 5,
    "cache_k": 6, "cache_v": 7, "query": 8, "sink": 9,
    "codes_k": 10, "codes_v": 11, "block_table": 12, "seq_lens": 13,
    "bench": 14, "new_k": 15, "new_v": 16, "scales_k": 17,
    "device_cache": 18,
}


@dataclass(frozen=True)
class Workload:
    """Shape and statistics of one synthetic workload."""
    name: str
    config_id: int
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    seq_len: int
    windows: Tuple[int, ...] = (0,)      # one entry per layer; 0 = full attention
    kv_alpha: float = 1.0
    q_alpha: float = 0.5
    q_basis_aligned: bool = True
    sinks: bool = False
    dtype: str = "bf16"                  # storage dtype of q, k, v ("f32" | "bf16")
    calib_tokens: int = 16384
    calib_config_id: Optional[int] = None  # reuse another workload's calibration seeds
    block_size: int = 0                  # 0 = contiguous cache, else paged block size
    n_new: int = 0                       # tokens appended per sequence (append workload)
    group_dim: int = 4
    codebook_size: int = 256

    @property
    def gqa(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def groups(self) -> int:
        return self.head_dim // self.group_dim

    @property
    def num_layers(self) -> int:
        return len(self.windows)

    @property
    def seed_config(self) -> int:
        return self.calib_config_id if self.calib_config_id is not None else self.config_id

    def code_bytes_per_step(self, layer: int = 0) -> int:
        """K + V code bytes read by one decode step of ``layer``."""
        w = self.windows[layer]
        attended = min(w, self.seq_len) if w > 0 else self.seq_len
        return 2 * self.batch * self.num_kv_heads * attended * self.groups

    def scaled(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    # Single head, batch 1, D=128, S=2048, fp32 inputs.
    "single_head": Workload("single_head", 1, batch=1, num_q_heads=1, num_kv_heads=1,
                            head_dim=128, seq_len=2048, dtype="f32"),
    # Qwen3-8B-shaped GQA decode layer.
    "qwen3_8b": Workload("qwen3_8b", 2, batch=8, num_q_heads=32, num_kv_heads=8,
                         head_dim=128, seq_len=16384),
    # Bandwidth sweep on the same shape (calibration shared with qwen3_8b).
    "sweep_b64_s32k": Workload("sweep_b64_s32k", 3, batch=64, num_q_heads=32, num_kv_heads=8,
                               head_dim=128, seq_len=32768, calib_config_id=2),
    "sweep_b1_s128k": Workload("sweep_b1_s128k", 3, batch=1, num_q_heads=32, num_kv_heads=8,
                               head_dim=128, seq_len=131072, calib_config_id=2),
    # GPT-OSS-20B-shaped layer pair: layer 0 sliding window 128, layer 1 full; sinks.
    "gptoss_pair": Workload("gptoss_pair", 4, batch=16, num_q_heads=64, num_kv_heads=8,
                            head_dim=64, seq_len=65536, windows=(128, 0), kv_alpha=2.0,
                            q_basis_aligned=False, sinks=True),
    # Append (4096 new tokens x 32 sequences, paged, 16-token blocks) then decode at 32768.
    "append_paged": Workload("append_paged", 5, batch=32, num_q_heads=32, num_kv_heads=8,
                             head_dim=128, seq_len=32768, calib_config_id=2,
                             block_size=16, n_new=4096),
}


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]


# --------------------------------------------------------------------------- RNG

def rng_for(config_id: int, layer: int, kv_head: int, role: str, index: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence([int(config_id), int(layer), int(kv_head), ROLE[role], int(index)])
    return np.random.Generator(np.random.PCG64(ss))


def haar_orthogonal(rng: np.random.Generator, d: int) -> np.ndarray:
    """Haar-distributed orthogonal matrix (QR of a Gaussian, signs fixed by diag(R))."""
    a = rng.standard_normal((d, d))
    q, r = np.linalg.qr(a)
    return q * np.sign(np.diag(r))[None, :]


def power_spectrum(d: int, alpha: float) -> np.ndarray:
    """lam_i proportional to i^-alpha (i = 1..d), scaled so that sum(lam) = d."""
    lam = np.arange(1, d + 1, dtype=np.float64) ** (-float(alpha))
    return lam * (d / lam.sum())


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even); returns float32."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Values exactly representable in the storage dtype, as float64."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return round_to_bf16(x).astype(np.float64)
    raise ValueError(dtype)


# ----------------------------------------------------------------- covariances

def head_bases(wl: Workload, layer: int, kv_head: int):
    """Orthogonal bases (U_k, U_v, U_q) of one (layer, KV head)."""
    c = wl.seed_config
    u_k = haar_orthogonal(rng_for(c, layer, kv_head, "basis_k"), wl.head_dim)
    u_v = haar_orthogonal(rng_for(c, layer, kv_head, "basis_v"), wl.head_dim)
    if wl.q_basis_aligned:
        u_q = u_k
    else:
        u_q = haar_orthogonal(rng_for(c, layer, kv_head, "basis_q"), wl.head_dim)
    return u_k, u_v, u_q


def _draw(rng: np.random.Generator, n: int, basis: np.ndarray, lam: np.ndarray) -> np.ndarray:
    z = rng.standard_normal((n, basis.shape[0]))
    return (z * np.sqrt(lam)[None, :]) @ basis.T


def calibration_set(wl: Workload, layer: int, kv_head: int, tokens: Optional[int] = None):
    """Calibration keys (M, D), values (M, D) and queries (G, M, D), storage-rounded."""
    m = wl.calib_tokens if tokens is None else tokens
    c = wl.seed_config
    d = wl.head_dim
    u_k, u_v, u_q = head_bases(wl, layer, kv_head)
    lam_kv = power_spectrum(d, wl.kv_alpha)
    lam_q = power_spectrum(d, wl.q_alpha)
    k = _draw(rng_for(c, layer, kv_head, "calib_k"), m, u_k, lam_kv)
    v = _draw(rng_for(c, layer, kv_head, "calib_v"), m, u_v, lam_kv)
    q = np.stack([_draw(rng_for(c, layer, kv_head, "calib_q", h), m, u_q, lam_q)
                  for h in range(wl.gqa)])
    return to_storage(k, wl.dtype), to_storage(v, wl.dtype), to_storage(q, wl.dtype)


def cache_tokens(wl: Workload, layer: int, kv_head: int, seq: int, n: int, start: int = 0):
    """Cached keys/values of positions [start, start+n) of sequence ``seq``: (n, D) each.

    Tokens are drawn in chunks of 1024 positions so that any sub-range is
    reproducible without drawing the whole sequence.
    """
    c = wl.config_id
    d = wl.head_dim
    u_k, u_v, _ = head_bases(wl, layer, kv_head)
    lam = power_spectrum(d, wl.kv_alpha)
    out_k = np.empty((n, d))
    out_v = np.empty((n, d))
    chunk = 1024
    t = start
    while t < start + n:
        ci = t // chunk
        lo = ci * chunk
        rk = rng_for(c, layer, kv_head, "cache_k", seq * 1_000_003 + ci)
        rv = rng_for(c, layer, kv_head, "cache_v", seq * 1_000_003 + ci)
        kk = _draw(rk, chunk, u_k, lam)
        vv = _draw(rv, chunk, u_v, lam)
        a = t - lo
        b = min(chunk, start + n - lo)
        out_k[t - start:t - start + (b - a)] = kk[a:b]
        out_v[t - start:t - start + (b - a)] = vv[a:b]
        t = lo + b
    return to_storage(out_k, wl.dtype), to_storage(out_v, wl.dtype)


def device_cache_tokens(wl: Workload, layer: int, seq: int, n: int, start: int, device):
    """Keys and values of positions [start, start+n) of sequence ``seq`` for
    every KV head, drawn on the device: two bf16 tensors [n][Hkv][D].

    The same statistical model as ``cache_tokens`` (the unit's Haar basis and
    power spectrum), with the Gaussian draws taken from torch's Philox
    generator on ``device`` instead of NumPy, so that long histories of many
    sequences are produced without host work.  The generator is seeded from
    (config, layer, seq, start) only, so a call is reproducible; it is not
    value-identical to ``cache_tokens``.  Draws and products are fp32, then
    rounded once to bf16 (nearest even).
    """
    import torch

    if wl.dtype != "bf16":
        raise ValueError("device_cache_tokens stores bf16")
    d, h = wl.head_dim, wl.num_kv_heads
    seed = int(np.random.SeedSequence([wl.config_id, layer, seq, start, ROLE["device_cache"]])
               .generate_state(1, dtype=np.uint64)[0] & 0x7FFFFFFFFFFFFFFF)
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    outs = []
    for side in (0, 1):
        # scaled basis per head: x = z diag(sqrt(lam)) U^T, as one [H][D][D] fp32 operand
        mats = np.stack([(np.sqrt(power_spectrum(d, wl.kv_alpha))[:, None] * head_bases(wl, layer, kv)[side].T)
                         for kv in range(h)])
        m = torch.as_tensor(mats, dtype=torch.float32).contiguous().to(device)
        z = torch.randn((h, n, d), generator=gen, device=device, dtype=torch.float32)
        x = torch.bmm(z, m)                                   # [H][n][D] fp32
        outs.append(x.transpose(0, 1).contiguous().to(torch.bfloat16))
    return outs[0], outs[1]


def decode_queries(wl: Workload, layer: int, batch: Optional[int] = None) -> np.ndarray:
    """Decode-step queries q[B][Hq][D], storage-rounded."""
    bsz = wl.batch if batch is None else batch
    d = wl.head_dim
    lam_q = power_spectrum(d, wl.q_alpha)
    q = np.empty((bsz, wl.num_q_heads, d))
    for kv in range(wl.num_kv_heads):
        _, _, u_q = head_bases(wl, layer, kv)
        for g in range(wl.gqa):
            h = kv * wl.gqa + g
            q[:, h, :] = _draw(rng_for(wl.config_id, layer, kv, "query", h), bsz, u_q, lam_q)
    return to_storage(q, wl.dtype)


def sink_logits(wl: Workload, layer: int) -> Optional[np.ndarray]:
    """Learned-sink stand-ins: one N(0,1) logit per query head (fp32), or None."""
    if not wl.sinks:
        return None
    s = rng_for(wl.config_id, layer, 0, "sink").standard_normal(wl.num_q_heads)
    return s.astype(np.float32).astype(np.float64)


def random_codes(wl: Workload, layer: int, side: str, shape) -> np.ndarray:
    """Uniform code bytes (a stand-in cache whose inputs need no encoding)."""
    role = "codes_k" if side == "k" else "codes_v"
    return rng_for(wl.config_id, layer, 0, role).integers(0, wl.codebook_size, size=shape,
                                                          dtype=np.uint8)


def random_key_scales(wl: Workload, layer: int, shape, sigma: float = 0.5) -> np.ndarray:
    """bf16 bit patterns (uint16) of log-normal positive values exp(N(0, sigma^2)):
    a stand-in pool of per-token key scales for a cache of random codes."""
    x = np.exp(sigma * rng_for(wl.config_id, layer, 0, "scales_k").standard_normal(shape))
    return (round_to_bf16(x).view(np.uint32) >> 16).astype(np.uint16)


def shuffled_block_table(wl: Workload, capacity_tokens: Optional[int] = None) -> np.ndarray:
    """Block table [B][blocks_per_seq] holding a seeded permutation of all physical blocks."""
    cap = wl.seq_len if capacity_tokens is None else capacity_tokens
    nb = cap // wl.block_size
    perm = rng_for(wl.config_id, 0, 0, "block_table").permutation(wl.batch * nb)
    return perm.reshape(wl.batch, nb).astype(np.int32)


def uniform_seq_lens(wl: Workload, lo: int, hi: int, index: int = 0) -> np.ndarray:
    """Sequence lengths drawn uniformly from [lo, hi] (ragged batches)."""
    return rng_for(wl.config_id, 0, 0, "seq_lens", index).integers(lo, hi + 1, size=wl.batch,
                                                                    dtype=np.int64).astype(np.int32)


def bench_params(wl: Workload, layer: int = 0):
    """Random transforms and codebooks of the right shapes and dtypes.

    The encode and decode kernels do the same work whatever these values are,
    so a throughput run can use them instead of a calibrated set: t_k is a
    Haar orthogonal matrix (its inverse transpose is itself), t_v another one,
    the codebooks are fp16 N(0, 1) draws and the key mean is small noise.
    """
    d, L, n = wl.head_dim, wl.groups, wl.codebook_size
    out = {"kbar": [], "t_k": [], "t_k_inv_t": [], "t_v": [], "cb_k": [], "cb_v": []}
    for kv in range(wl.num_kv_heads):
        r = rng_for(wl.config_id, layer, kv, "bench")
        qk = haar_orthogonal(r, d).astype(np.float32)
        out["t_k"].append(qk)
        out["t_k_inv_t"].append(qk.copy())
        out["t_v"].append(haar_orthogonal(r, d).astype(np.float32))
        out["kbar"].append((0.1 * r.standard_normal(d)).astype(np.float32))
        out["cb_k"].append(r.standard_normal((L, n, wl.group_dim)).astype(np.float16))
        out["cb_v"].append(r.standard_normal((L, n, wl.group_dim)).astype(np.float16))
    return {k: np.stack(v) for k, v in out.items()}
