"""Throughput of the NOVA-KV hot path on one MI355X.

One step = the whole hot path for one decode step of the Qwen3-8B-shaped
layer (32 query / 8 KV heads, head_dim 128, batch 8, context 16384, 2-bit VQ
K and V caches): nova_kv_append_decode_attn, one launch that encodes the
step's new key/value (one token per sequence, stored at position S-1) and
runs decode attention of one query per head over all S cached tokens.  The
same step as two calls (nova_kv_encode, then nova_kv_decode_attn) is timed
beside it, and each of those kernels alone.
Inputs are resident in HBM before timing; the code pools rotate over six
copies (6 x 64 MiB) so the 256 MB last-level cache cannot serve them.

Printed metric: effective compressed-KV bandwidth = K+V code bytes attended
per step / time per step, with microseconds per step and the fraction of the
8 TB/s HBM peak beside it.  A CPU baseline (the fp64 oracle on host cores, a
bounded sample of the same workload) is reported next to it.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
WORKLOAD = "qwen3_8b"
COPIES = 6
DECODE_KERNEL = "decode_lut_d128"
# The step kernel's source and the headers it includes: a change to any of
# them invalidates the committed counter summary.
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_04074_amd", "csrc", f)
                  for f in ("decode_lut.hip", "band_attention.h", "encode_block.h", "lut_common.h",
                            "nova_kv_internal.h")]
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "decode_lut_d128_qwen3_8b_traffic.md")
COPY_CALIB_BYTES = 256 << 20


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=1000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time budget of the oracle baseline sample")
    ap.add_argument("--skip-append", action="store_true")
    ap.add_argument("--skip-others", action="store_true",
                    help="do not time the decode of the other workload shapes")
    ap.add_argument("--copy-calib", action="store_true",
                    help=f"finish with one plain device copy of {COPY_CALIB_BYTES >> 20} MiB, the known-size "
                         "reference for scaling FETCH_SIZE / WRITE_SIZE counter runs")
    return ap.parse_args()


def kernel_source_sha256() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(os.path.basename(path).encode() + b"\0" + f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per decode launch from the committed counter summary, or None
    when the summary is missing or was taken on a different kernel source."""
    try:
        text = open(TRAFFIC_SUMMARY).read()
    except OSError:
        return None
    sha = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9]+)", text)
    if not sha or not val or sha.group(1) != kernel_source_sha256():
        return None
    return int(val.group(1))


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


def other_workloads(nk, torch, dev, calls: int):
    """Decode-kernel time of every other workload shape (one line each).

    Pools hold uniformly random codes (and, in the key-scale format, random
    bf16 scales); shapes too small to exceed the 256 MB last-level cache are
    measured as they would run (cache-resident)."""
    import synth
    res = []
    # (workload, layer, key-scale format, sink-plus-recent band (n_sink, n_rec) or None,
    #  fp8 codebooks, scalar value arm)
    cases = [("single_head", 0, False, None, False, False), ("sweep_b64_s32k", 0, False, None, False, False),
             ("sweep_b1_s128k", 0, False, None, False, False), ("gptoss_pair", 0, False, None, False, False),
             ("gptoss_pair", 1, False, None, False, False), ("append_paged", 0, False, None, False, False),
             ("qwen3_8b", 0, True, None, False, False), ("gptoss_pair", 1, True, None, False, False),
             ("qwen3_8b", 0, False, (64, 256), False, False), ("gptoss_pair", 1, False, (64, 256), False, False),
             ("qwen3_8b", 0, False, None, True, False), ("gptoss_pair", 1, False, None, True, False),
             ("qwen3_8b", 0, False, None, False, True)]
    for name, layer, key_scale, band_sizes, fp8, sq in cases:
        wl = synth.get_workload(name)
        B, S, H, Hq, D, L = wl.batch, wl.seq_len, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.groups
        gen = torch.Generator(device=dev)
        gen.manual_seed(7)
        arrays = synth.bench_params(wl, layer)
        if fp8:  # the same codebooks rounded to fp8 E4M3 (torch's conversion), as bytes
            for k in ("cb_k", "cb_v"):
                arrays[k] = torch.as_tensor(arrays[k]).to(torch.float32).to(torch.float8_e4m3fn).view(torch.uint8)
        P = nk.NovaKVParams.from_arrays(arrays, device=dev, key_scale=key_scale, sq_values=sq)
        if wl.block_size:
            bps = S // wl.block_size
            layout = nk.CacheLayout(wl.block_size, bps, torch.as_tensor(synth.shuffled_block_table(wl)).to(dev))
            shape = (B * bps, H, wl.block_size, L)
        else:
            layout = nk.CacheLayout.contiguous(S)
            shape = (B, H, S, L)
        scale_bytes = 2 * int(np.prod(shape[:3])) if key_scale else 0
        pool_bytes = 2 * int(np.prod(shape)) + scale_bytes
        copies = int(min(6, max(1, -(-(600 << 20) // pool_bytes)))) if pool_bytes > (64 << 20) else 1
        pools = [(torch.randint(0, 256, shape, dtype=torch.uint8, device=dev, generator=gen),
                  torch.randint(0, 256, shape, dtype=torch.uint8, device=dev, generator=gen),
                  (torch.rand(shape[:3], generator=gen, device=dev) + 0.5).to(torch.bfloat16)
                  if key_scale else None,
                  torch.randn(shape[:3] + (2,), generator=gen, device=dev).to(torch.bfloat16) if sq else None)
                 for _ in range(copies)]
        q = torch.randn((B, Hq, D), generator=gen, device=dev).to(torch.bfloat16)
        seq = torch.full((B,), S, dtype=torch.int32, device=dev)
        sinks = torch.as_tensor(synth.sink_logits(wl, layer), dtype=torch.float32).to(dev) if wl.sinks else None
        out = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
        ws = torch.zeros(nk.decode_workspace_bytes(P, B, Hq, S), dtype=torch.uint8, device=dev)
        window = wl.windows[layer]
        band = None
        if band_sizes:
            bshape = nk.band_shape(P, B, *band_sizes)
            band = nk.Band(*band_sizes, torch.randn(bshape, generator=gen, device=dev).to(torch.bfloat16),
                           torch.randn(bshape, generator=gen, device=dev).to(torch.bfloat16))
        calls_ = [nk.prepare_decode(P, layout, q, pk, pv, seq, S, out, ws, window=window, sinks=sinks,
                                    k_scales=ps, band=band, v_sq=pq)
                  for pk, pv, ps, pq in pools]
        for i in range(5):
            calls_[i % copies]()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(calls):
            calls_[i % copies]()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / calls
        cb = wl.code_bytes_per_step(layer)
        bb = 0
        if band_sizes:  # the band's tokens are read as bf16 rows instead of codes
            nband = min(sum(band_sizes), S)
            cb -= 2 * B * H * nband * L
            bb = 2 * B * H * nband * D * 2
        # the key scales of the tokens read from codes: 2 bytes per token and KV
        # head; the value scale and offset: 4 more
        sb = (cb // L if key_scale else 0) + (2 * cb // L if sq else 0)
        res.append({"workload": f"{name}" + (f" layer {layer} (window {window})" if wl.num_layers > 1 else "")
                    + (" key-scale format" if key_scale else "")
                    + (f" band {band_sizes[0]}+{band_sizes[1]}" if band_sizes else "")
                    + (" fp8 codebooks" if fp8 else "")
                    + (" scalar value arm" if sq else ""),
                    "batch": B, "seq_len": S, "q_heads": Hq, "kv_heads": H, "head_dim": D,
                    "paged_block": wl.block_size or None, "code_bytes": cb, "scale_bytes": sb,
                    "band_bytes": bb, "pool_copies": copies,
                    "decode_us": round(us, 2), "GB_per_s": round((cb + sb + bb) / (us * 1e-6) / 1e9, 1),
                    "frac_of_hbm_peak": round((cb + sb + bb) / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)})
        del pools, calls_, ws, band
        torch.cuda.empty_cache()
    return res


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

    # prepared calls: arguments marshalled once, so the host keeps ahead of the GPU
    enc_calls = [nk.prepare_encode(P, layout, k_new, v_new, start_pos, pk, pv) for pk, pv in pools]
    dec_calls = [nk.prepare_decode(P, layout, q, pk, pv, seq_lens, S, out, ws) for pk, pv in pools]
    step_calls = [nk.prepare_append_decode(P, layout, k_new[:, 0], v_new[:, 0], q, pk, pv, seq_lens, S, out, ws)
                  for pk, pv in pools]

    def step(i):
        step_calls[i % COPIES]()

    def two_call_step(i):
        enc_calls[i % COPIES]()
        dec_calls[i % COPIES]()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    def timed(fn, n):
        """Mean GPU time per call of n back-to-back calls, events on the current
        stream (the stream the calls launch on)."""
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for i in range(n):
            fn(i)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / n

    # whole step (append the new token and decode attention, one launch): the headline
    ms_step = timed(step, args.steps) * 1e-3
    step_runs = [timed(step, args.steps) for _ in range(5)]
    two_call_us = timed(two_call_step, args.steps)
    # each kernel alone, back to back, for the roofline of the dominant kernel
    n_runs = 5
    dec_runs = [timed(lambda i: dec_calls[i % COPIES](), args.steps) for _ in range(n_runs)]
    enc_runs = [timed(lambda i: enc_calls[i % COPIES](), args.steps) for _ in range(n_runs)]
    dec_mean_us = float(np.mean(dec_runs))
    dec_med_us = float(np.median(dec_runs))
    enc_us = np.array(enc_runs)
    # the same step with the codebooks in the paper's stored format: rounded to
    # fp8 E4M3 (torch's conversion) and passed as bytes
    p8 = dict(params)
    for k in ("cb_k", "cb_v"):
        p8[k] = torch.as_tensor(params[k]).to(torch.float32).to(torch.float8_e4m3fn).view(torch.uint8)
    P8 = nk.NovaKVParams.from_arrays(p8, device=dev)
    step8_calls = [nk.prepare_append_decode(P8, layout, k_new[:, 0], v_new[:, 0], q, pk, pv, seq_lens, S, out, ws)
                   for pk, pv in pools]
    for i in range(200):
        step8_calls[i % COPIES]()
    step8_runs = [timed(lambda i: step8_calls[i % COPIES](), args.steps) for _ in range(n_runs)]

    value = code_bytes / (ms_step * 1e-3) / 1e9
    step_mean_us = float(np.mean(step_runs))
    achieved = code_bytes / (step_mean_us * 1e-6) / 1e9

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

    others = None if args.skip_others else other_workloads(nk, torch, dev, 50)

    if args.copy_calib:  # plain copy of known size, last dispatch of the run
        src = torch.empty(COPY_CALIB_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, args.cpu_seconds)
    traffic = measured_traffic()

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
                        "per sequence + decode attention, one launch",
            "batch": B, "seq_len": S, "q_heads": Hq, "kv_heads": H, "head_dim": D,
            "code_bytes_per_step": code_bytes, "pool_copies": COPIES,
            "params": "random orthogonal transforms, fp16 N(0,1) codebooks, uniform random codes",
        },
        "step_kernel_us": {"mean": round(step_mean_us, 2),
                           "median_of_runs": round(float(np.median(step_runs)), 2),
                           "min_of_runs": round(float(np.min(step_runs)), 2),
                           "max_of_runs": round(float(np.max(step_runs)), 2),
                           "runs": len(step_runs), "calls_per_run": args.steps},
        "step_fp8_codebooks_us": {"mean": round(float(np.mean(step8_runs)), 2),
                                  "median_of_runs": round(float(np.median(step8_runs)), 2)},
        "two_call_step_us": round(two_call_us, 2),
        "decode_kernel_us": {"mean": round(dec_mean_us, 2), "median_of_runs": round(dec_med_us, 2),
                             "min_of_runs": round(float(np.min(dec_runs)), 2),
                             "max_of_runs": round(float(np.max(dec_runs)), 2),
                             "runs": n_runs, "calls_per_run": args.steps},
        "append_kernel_us": {"mean": round(float(np.mean(enc_us)), 2),
                             "median_of_runs": round(float(np.median(enc_us)), 2)},
        "roofline": {
            "kernel": f"{DECODE_KERNEL}<12, true, false, false, false> (the step's one launch: encode of the new token, query "
                      "transform, split pass, combine)",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": code_bytes,
        },
        "append_encode": append,
        "other_workloads_decode": others,
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
