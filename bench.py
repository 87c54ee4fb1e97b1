"""Throughput of the NOVA-KV hot path on one MI355X.

One step = the whole hot path for one decode step of the Qwen3-8B-shaped
layer (32 query / 8 KV heads, head_dim 128, batch 8, context 16384, 2-bit VQ
K and V caches):
  1. nova_kv_encode of the step's new key/value (one token per sequence,
     appended at position S-1), then
  2. nova_kv_decode_attn of one query per head over all S cached tokens.
Inputs are resident in HBM before timing; the code pools rotate over six
copies (6 x 64 MiB) so the 256 MB last-level cache cannot serve them.

Printed metric: effective compressed-KV bandwidth = K+V code bytes attended
per step / time per step, with microseconds per step and the fraction of the
8 TB/s HBM peak beside it.  A CPU baseline (the fp64 oracle on host cores, a
bounded sample of the same workload) is reported next to it.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
WORKLOAD = "qwen3_8b"
COPIES = 6


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time budget of the oracle baseline sample")
    ap.add_argument("--skip-append", action="store_true")
    return ap.parse_args()


def cpu_baseline(wl, budget_s: float):
    """Time the fp64 oracle (plain-form decode + encode of the new token) on sampled units."""
    from oracle import attention as oatt
    from oracle import codec as ocodec
    import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    params = synth.bench_params(wl)
    S, L, G, D = wl.seq_len, wl.groups, wl.gqa, wl.head_dim
    q = synth.decode_queries(wl, 0)
    scale = 1.0 / np.sqrt(D)
    rng = np.random.default_rng(0)
    units = [(b, kv) for b in range(wl.batch) for kv in range(wl.num_kv_heads)]
    done = 0
    t0 = time.perf_counter()
    elapsed = 0.0
    while done < len(units) and (elapsed < budget_s or done == 0):
        b, kv = units[done]
        hp = oatt.head_params(params, kv)
        ck = rng.integers(0, 256, (S, L), dtype=np.uint8)
        cv = rng.integers(0, 256, (S, L), dtype=np.uint8)
        kn, vn = synth.cache_tokens(wl, 0, kv, b, 1, start=S - 1)
        t1 = time.perf_counter()
        nk_, _, nv_, _ = ocodec.encode_tokens(kn, vn, hp)
        ck[-1], cv[-1] = nk_[0], nv_[0]
        oatt.decode_rows(q[b, kv * G:(kv + 1) * G], ck, cv, hp, scale)
        elapsed += time.perf_counter() - t1
        done += 1
    per_unit = elapsed / done
    step_s = per_unit * len(units)
    code_bytes = wl.code_bytes_per_step()
    return {
        "value": round(code_bytes / step_s / 1e9, 4),
        "unit": "GB/s",
        "us_per_step": round(step_s * 1e6, 1),
        "cores": int(threads),
        "host_cpus": os.cpu_count(),
        "kind": "oracle",
        "sample": f"{done} of {len(units)} (sequence, KV head) units: encode 1 token + plain-form "
                  f"fp64 decode of {G} heads over {S} tokens each; step time = mean unit time x "
                  f"{len(units)}",
        "wall_s": round(time.perf_counter() - t0, 2),
    }


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(the decode shards by KV head with no exchange; see the design notes).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2608_04074_amd as nk
    import synth

    wl = synth.get_workload(WORKLOAD)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B, S, H, Hq, D, L = wl.batch, wl.seq_len, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.groups
    code_bytes = wl.code_bytes_per_step()

    params = synth.bench_params(wl)
    P = nk.NovaKVParams.from_arrays(params, device=dev)
    layout = nk.CacheLayout.contiguous(S)
    gen = torch.Generator(device=dev)
    gen.manual_seed(1234)
    pools = []
    for _ in range(COPIES):
        pk = torch.randint(0, 256, (B, H, S, L), dtype=torch.uint8, device=dev, generator=gen)
        pv = torch.randint(0, 256, (B, H, S, L), dtype=torch.uint8, device=dev, generator=gen)
        pools.append((pk, pv))
    q = torch.as_tensor(synth.decode_queries(wl, 0)).to(torch.bfloat16).to(dev)
    k_new = torch.randn((B, 1, H, D), generator=gen, device=dev).to(torch.bfloat16)
    v_new = torch.randn((B, 1, H, D), generator=gen, device=dev).to(torch.bfloat16)
    start_pos = torch.full((B,), S - 1, dtype=torch.int32, device=dev)
    seq_lens = torch.full((B,), S, dtype=torch.int32, device=dev)
    out = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
    ws = torch.zeros(nk.decode_workspace_bytes(P, B, Hq, S), dtype=torch.uint8, device=dev)

    def step(i, ev=None):
        pk, pv = pools[i % COPIES]
        nk.encode(P, layout, k_new, v_new, start_pos, pk, pv)
        if ev is not None:
            ev[0].record()
        nk.decode_attn(P, layout, q, pk, pv, seq_lens, S, out=out, workspace=ws)
        if ev is not None:
            ev[1].record()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        step(i, evs[i])
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_step = total_ms / args.steps
    dec_ms = np.array([a.elapsed_time(b) for a, b in evs])
    dec_med_us = float(np.median(dec_ms) * 1e3)
    dec_mean_us = float(np.mean(dec_ms) * 1e3)

    value = code_bytes / (ms_step * 1e-3) / 1e9
    achieved = code_bytes / (dec_mean_us * 1e-6) / 1e9

    # Append throughput (prefill-encode of 4096 tokens x 32 sequences x 8 KV heads), reported aside.
    append = None
    if not args.skip_append:
        awl = synth.get_workload("append_paged")
        kk = torch.randn((awl.batch, awl.n_new, H, D), generator=gen, device=dev).to(torch.bfloat16)
        vv = torch.randn((awl.batch, awl.n_new, H, D), generator=gen, device=dev).to(torch.bfloat16)
        bps = awl.seq_len // awl.block_size
        table = torch.as_tensor(synth.shuffled_block_table(awl)).to(dev)
        alay = nk.CacheLayout(awl.block_size, bps, table)
        apk = torch.zeros((awl.batch * bps, H, awl.block_size, L), dtype=torch.uint8, device=dev)
        apv = torch.zeros_like(apk)
        sp = torch.full((awl.batch,), awl.seq_len - awl.n_new, dtype=torch.int32, device=dev)
        nk.encode(P, alay, kk, vv, sp, apk, apv)
        torch.cuda.synchronize()
        reps = 3
        a0 = torch.cuda.Event(enable_timing=True)
        a1 = torch.cuda.Event(enable_timing=True)
        a0.record()
        for _ in range(reps):
            nk.encode(P, alay, kk, vv, sp, apk, apv)
        a1.record()
        torch.cuda.synchronize()
        a_ms = a0.elapsed_time(a1) / reps
        th = awl.batch * awl.n_new * H
        append = {"workload": "append 4096 tokens x 32 sequences, 8 KV heads, D=128, paged 16-token blocks",
                  "ms": round(a_ms, 3), "token_heads_per_s": round(th / (a_ms * 1e-3), 1)}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, args.cpu_seconds)

    rec = {
        "metric": "VQ-KV decode attention effective compressed-KV bandwidth (K+V code bytes / step time), S=16K",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "us_per_step": round(ms_step * 1e3, 2),
        "frac_of_hbm_peak": round(value / HBM_PEAK_GBS, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "qwen3_8b-shaped GQA decode layer over a 2-bit VQ K/V cache: encode 1 new token "
                        "per sequence + decode attention",
            "batch": B, "seq_len": S, "q_heads": Hq, "kv_heads": H, "head_dim": D,
            "code_bytes_per_step": code_bytes, "pool_copies": COPIES,
            "params": "random orthogonal transforms, fp16 N(0,1) codebooks, uniform random codes",
        },
        "decode_call_us": {"median": round(dec_med_us, 2), "mean": round(dec_mean_us, 2)},
        "roofline": {
            "kernel": "decode call (prologue + stage 1 + combine)",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None,
        },
        "append_encode": append,
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
