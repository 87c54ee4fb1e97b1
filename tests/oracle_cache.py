"""Oracle calibrations of the synthetic workloads, cached on disk.

Calibration (Algorithms 2 and 3) is the slow part of the oracle, and its
outputs are inputs of the GPU path.  This module runs it through ``oracle/``
only and keeps the results in ``tests/_cache/`` (not committed) keyed by
workload, layer and calibration settings, so repeated test sessions reuse
them.  Deleting the cache only costs time.
"""

from __future__ import annotations

import hashlib
import json
import os

import numpy as np

import synth
from oracle import calibration
from oracle import fp8 as oracle_fp8

CACHE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_cache")
KEYS = ("kbar", "t_k", "t_k_inv_t", "t_v", "cb_k", "cb_v")
VERSION = 1


def _key(wl: synth.Workload, layer: int, tokens: int, iters: int, mo_stride: int,
         key_scale: bool = False) -> str:
    fields = [VERSION, wl.seed_config, wl.num_q_heads, wl.num_kv_heads, wl.head_dim,
              wl.kv_alpha, wl.q_alpha, wl.q_basis_aligned, wl.dtype, layer, tokens,
              iters, mo_stride]
    if key_scale:
        fields.append("key_scale")
    desc = json.dumps(fields)
    return hashlib.sha1(desc.encode()).hexdigest()[:16]


def calibrated_params(wl: synth.Workload, layer: int = 0, tokens: int = None, iters: int = 25,
                      mo_stride: int = 16, heads=None, key_scale: bool = False, fp8: bool = False):
    """Stacked [Hkv][...] stored parameters of one layer (oracle calibration per KV head).

    key_scale: key codebooks trained on normalized coefficients (key-scale format).
    fp8: the fp16 codebooks snapped to fp8 E4M3 (still held as fp16 values)."""
    tokens = wl.calib_tokens if tokens is None else tokens
    heads = range(wl.num_kv_heads) if heads is None else heads
    os.makedirs(CACHE, exist_ok=True)
    per_head = []
    for kv in heads:
        path = os.path.join(CACHE, f"{wl.name}_L{layer}_kv{kv}_{_key(wl, layer, tokens, iters, mo_stride, key_scale)}.npz")
        if os.path.exists(path):
            with np.load(path, allow_pickle=False) as z:
                per_head.append({k: z[k] for k in KEYS})
            continue
        k, v, q = synth.calibration_set(wl, layer, kv, tokens)
        stored, _ = calibration.calibrate_head(k, v, q, mo_stride=mo_stride, kmeans_iters=iters,
                                               seed=[wl.seed_config, layer, kv], key_scale=key_scale)
        np.savez(path + ".tmp.npz", **stored)
        os.replace(path + ".tmp.npz", path)
        per_head.append(stored)
    out = calibration.stack_params(per_head)
    if fp8:
        out = dict(out, cb_k=oracle_fp8.snap_codebooks(out["cb_k"]), cb_v=oracle_fp8.snap_codebooks(out["cb_v"]))
    return out


if __name__ == "__main__":
    import sys
    import time
    names = sys.argv[1:] or ["single_head", "qwen3_8b", "gptoss_pair"]
    for name in names:
        wl = synth.get_workload(name)
        for layer in range(wl.num_layers):
            t = time.time()
            calibrated_params(wl, layer)
            print(f"{name} layer {layer}: {time.time() - t:.1f}s", flush=True)
