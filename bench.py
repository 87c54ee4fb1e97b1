"""Throughput of the NOVA-KV hot path on one MI355X.

One step = the whole hot path for one decode step of the Qwen3-8B-shaped
layer (32 query / 8 KV heads, head_dim 128, batch 8, context 16384, 2-bit VQ
K and V caches): nova_kv_append_decode_attn, one launch that encodes the
step's new key/value (one token per sequence, stored at position S-1) and
runs decode attention of one query per head over all S cached tokens.  The
same step as two calls (nova_kv_encode, then nova_kv_decode_attn) is timed
beside it, and each of those kernels alone.
Inputs are resident in HBM before timing.  Every code pool of 16 MiB or more
rotates over enough copies (at least 600 MiB in all) that the 256 MB
last-level cache cannot serve it.

Printed metric: effective compressed-KV bandwidth = K+V code bytes attended
per step / time per step, with microseconds per step and the fraction of the
8 TB/s HBM peak beside it.  A CPU baseline (the fp64 oracle on host cores, a
bounded sample of the same workload, one process per core) is reported next
to it.
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
FP64_MFMA_PEAK_TFLOPS = 78.6
WORKLOAD = "qwen3_8b"
ROTATE_MIN_BYTES = 16 << 20       # pools this large rotate over copies ...
ROTATE_TOTAL_BYTES = 600 << 20    # ... until the copies hold at least this much
DECODE_KERNEL = "decode_lut_d128"
# The step kernel's source and the headers it includes: a change to any of
# them invalidates the committed counter summary.
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_04074_amd", "csrc", f)
                  for f in ("decode_lut.hip", "band_attention.h", "encode_block.h", "lut_common.h",
                            "nova_kv_internal.h")]
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "decode_lut_d128_qwen3_8b_traffic.md")
COUNTER_SUMMARY = os.path.join(ROOT, "profiles", "decode_lut_d128_qwen3_8b_counters.md")
COPY_CALIB_BYTES = 256 << 20
# Algorithmic work of the append encoder per token-head (D = 128, two sides):
# the transform (2 D^2 flops per side) and the exhaustive distances
# (2 * 256 * D flops per side: one multiply-add per codeword coordinate).
ENCODE_FLOPS_PER_TOKEN_HEAD = 2 * (2 * 128 * 128) + 2 * (2 * 256 * 128)

# Other workload lines: (name, layer, key-scale format, band (n_sink, n_rec) or
# None, fp8 codebooks, scalar value arm).
OTHER_CASES = [("single_head", 0, False, None, False, False), ("sweep_b64_s32k", 0, False, None, False, False),
               ("sweep_b1_s128k", 0, False, None, False, False), ("gptoss_pair", 0, False, None, False, False),
               ("gptoss_pair", 1, False, None, False, False), ("append_paged", 0, False, None, False, False),
               ("qwen3_8b", 0, True, None, False, False), ("gptoss_pair", 1, True, None, False, False),
               ("qwen3_8b", 0, False, (64, 256), False, False), ("gptoss_pair", 1, False, (64, 256), False, False),
               ("qwen3_8b", 0, False, None, True, False), ("gptoss_pair", 1, False, None, True, False),
               ("qwen3_8b", 0, False, None, False, True),
               # the deployed format: key scale, INT2 values, a 64+256 band
               ("qwen3_8b", 0, True, (64, 256), False, True), ("gptoss_pair", 1, True, (64, 256), False, True)]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=1000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate wall time of the oracle baseline sample")
    ap.add_argument("--skip-append", action="store_true")
    ap.add_argument("--skip-others", action="store_true",
                    help="do not time the decode of the other workload shapes")
    ap.add_argument("--only", default=None,
                    help="time one line only and skip the headline: an other-workload label prefix "
                         "(e.g. 'sweep_b1_s128k', 'gptoss_pair layer 1'), or 'append_encode'")
    ap.add_argument("--calls", type=int, default=200, help="timed calls per other-workload line")
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


def measured_counters():
    """The step kernel's SQ counter ratios from the committed summary (VALU issue
    and LDS issue per wave time, MFMA busy per SIMD time, LDS bank-conflict cycles
    per CU time), or None when it is missing or was taken on a different source."""
    try:
        text = open(COUNTER_SUMMARY).read()
    except OSError:
        return None
    sha = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    row = re.search(r"\| `" + re.escape(DECODE_KERNEL) + r"<12, true, false, false, false, false, false>` \| (\d+) \| ([0-9.]+) \| "
                    r"([0-9.]+) \| ([0-9.]+) \| ([0-9.]+) \| ([0-9.]+) \|", text)
    if not sha or not row or sha.group(1) != kernel_source_sha256():
        return None
    return {"source": os.path.relpath(COUNTER_SUMMARY, ROOT), "valu_issue_frac": float(row.group(3)),
            "mfma_busy_frac": float(row.group(4)), "lds_issue_frac": float(row.group(5)),
            "lds_bank_conflict_frac": float(row.group(6))}


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


def rotation_copies(pool_bytes: int, at_least: int = 1) -> int:
    """Copies of a pool so that a rotation over them defeats the last-level cache."""
    if pool_bytes < ROTATE_MIN_BYTES:
        return at_least
    return max(at_least, -(-ROTATE_TOTAL_BYTES // pool_bytes))


# ------------------------------------------------------------------ CPU baseline

def _cpu_unit(task):
    """One (sequence, KV head) unit of the step in the oracle: encode the new
    token, then the plain-form fp64 decode of the G heads over S tokens.
    Runs in a worker process with one BLAS/OpenMP thread."""
    b, kv = task
    from oracle import attention as oatt
    from oracle import codec as ocodec
    import synth
    wl = synth.get_workload(WORKLOAD)
    params = _cpu_unit.params
    S, L, G = wl.seq_len, wl.groups, wl.gqa
    rng = np.random.default_rng([b, kv])
    ck = rng.integers(0, 256, (S, L), dtype=np.uint8)
    cv = rng.integers(0, 256, (S, L), dtype=np.uint8)
    kn, vn = synth.cache_tokens(wl, 0, kv, b, 1, start=S - 1)
    hp = oatt.head_params(params, kv)
    q = _cpu_unit.q
    t0 = time.perf_counter()
    nk_, _, nv_, _ = ocodec.encode_tokens(kn, vn, hp)
    ck[-1], cv[-1] = nk_[0], nv_[0]
    oatt.decode_rows(q[b, kv * G:(kv + 1) * G], ck, cv, hp, 1.0 / np.sqrt(wl.head_dim))
    return time.perf_counter() - t0


def _cpu_worker_init():
    import synth
    wl = synth.get_workload(WORKLOAD)
    _cpu_unit.params = synth.bench_params(wl)
    _cpu_unit.q = synth.decode_queries(wl, 0)


def cpu_baseline(budget_s: float):
    """The oracle on the host cores: one worker process per core, each with one
    BLAS/OpenMP thread, over a bounded sample of the step's (sequence, KV head)
    units; the step time is the sample's wall time scaled to all units."""
    import multiprocessing as mp
    import synth
    wl = synth.get_workload(WORKLOAD)
    units = [(b, kv) for b in range(wl.batch) for kv in range(wl.num_kv_heads)]
    workers = max(1, min(len(units), os.cpu_count() or 1, 16))
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS", "BLIS_NUM_THREADS"):
        os.environ[var] = "1"
    ctx = mp.get_context("spawn")
    with ctx.Pool(workers, initializer=_cpu_worker_init) as pool:
        # one round of one unit per worker sizes the sample to the budget
        t0 = time.perf_counter()
        first = pool.map(_cpu_unit, units[:workers], chunksize=1)
        round_s = time.perf_counter() - t0
        rounds = int(max(0, min(len(units) // workers - 1, budget_s / max(round_s, 1e-3) - 1)))
        rest = units[workers:workers * (1 + rounds)]
        t1 = time.perf_counter()
        more = pool.map(_cpu_unit, rest, chunksize=1) if rest else []
        wall = time.perf_counter() - t1
    done = len(first) + len(more)
    # steady-state rate from the rounds after the first (which includes worker start-up)
    if more:
        rate = len(more) / wall
    else:
        rate = len(first) / round_s
    step_s = len(units) / rate
    code_bytes = wl.code_bytes_per_step()
    return {
        "value": round(code_bytes / step_s / 1e9, 4),
        "unit": "GB/s",
        "us_per_step": round(step_s * 1e6, 1),
        "cores": workers,
        "host_cpus": os.cpu_count(),
        "kind": "oracle",
        "sample": f"{done} of {len(units)} (sequence, KV head) units of the step, {workers} worker processes "
                  f"with one BLAS/OpenMP thread each: encode of the new token + plain-form fp64 decode of "
                  f"{wl.gqa} heads over {wl.seq_len} tokens per unit; step time = all {len(units)} units at "
                  f"the sample's unit rate",
        "unit_compute_s_mean": round(float(np.mean(first + more)), 4),
    }


# ------------------------------------------------------------------ GPU timing

def timed_calls(torch, fn, n: int):
    """Per-call GPU times (us) of n calls: an event before each call and one after
    the last, on the stream the calls launch on (torch's current stream)."""
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    torch.cuda.synchronize()
    for i in range(n):
        ev[i].record()
        fn(i)
    ev[n].record()
    torch.cuda.synchronize()
    return np.array([ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(n)])


def back_to_back_us(torch, fn, n: int) -> float:
    """Mean GPU time per call of n back-to-back calls (events around all of them)."""
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(n):
        fn(i)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / n


def pct(x):
    return {"p10": round(float(np.percentile(x, 10)), 2), "p50": round(float(np.percentile(x, 50)), 2),
            "p90": round(float(np.percentile(x, 90)), 2), "calls": int(len(x))}


def case_label(name, layer, key_scale, band_sizes, fp8, sq, wl):
    return (f"{name}" + (f" layer {layer} (window {wl.windows[layer]})" if wl.num_layers > 1 else "")
            + (" key-scale format" if key_scale else "")
            + (f" band {band_sizes[0]}+{band_sizes[1]}" if band_sizes else "")
            + (" fp8 codebooks" if fp8 else "")
            + (" scalar value arm" if sq else ""))


def other_workload(nk, torch, dev, case, calls: int):
    """Decode-kernel time of one workload shape (uniformly random codes; in the
    key-scale format random bf16 scales), pools rotated over copies."""
    import synth
    name, layer, key_scale, band_sizes, fp8, sq = case
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
    sq_bytes = 4 * int(np.prod(shape[:3])) if sq else 0
    pool_bytes = 2 * int(np.prod(shape)) + scale_bytes + sq_bytes
    copies = rotation_copies(pool_bytes)
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
    band, band_copies = None, 1
    bands = [None]
    if band_sizes:
        bshape = nk.band_shape(P, B, *band_sizes)
        band_bytes_all = 2 * 2 * int(np.prod(bshape))
        band_copies = max(1, min(copies, rotation_copies(band_bytes_all)))
        bands = [nk.Band(*band_sizes, torch.randn(bshape, generator=gen, device=dev).to(torch.bfloat16),
                         torch.randn(bshape, generator=gen, device=dev).to(torch.bfloat16))
                 for _ in range(band_copies)]
    calls_ = [nk.prepare_decode(P, layout, q, pk, pv, seq, S, out, ws, window=window, sinks=sinks,
                                k_scales=ps, band=bands[i % len(bands)], v_sq=pq)
              for i, (pk, pv, ps, pq) in enumerate(pools)]
    fn = lambda i: calls_[i % copies]()  # noqa: E731
    for i in range(200):
        fn(i)
    us = back_to_back_us(torch, fn, calls)
    per_call = timed_calls(torch, fn, calls)
    cb = wl.code_bytes_per_step(layer)
    bb = 0
    if band_sizes:  # the band's tokens are read as bf16 rows instead of codes
        nband = min(sum(band_sizes), S)
        cb -= 2 * B * H * nband * L
        bb = 2 * B * H * nband * D * 2
    # the key scales of the tokens read from codes: 2 bytes per token and KV
    # head; the value scale and offset: 4 more
    sb = (cb // L if key_scale else 0) + (2 * cb // L if sq else 0)
    step = {}
    if band_sizes:
        # the whole step on the same pools: append a token at seq_len - 1, then
        # attend; one launch on the table kernels when the band's recent part
        # holds the new token (it is then the band's last row)
        kn = torch.randn((B, H, D), generator=gen, device=dev).to(torch.bfloat16)
        vn = torch.randn((B, H, D), generator=gen, device=dev).to(torch.bfloat16)
        steps_ = [nk.prepare_append_decode(P, layout, kn, vn, q, pk, pv, seq, S, out, ws, window=window,
                                           sinks=sinks, k_scales=ps, band=bands[i % len(bands)], v_sq=pq)
                  for i, (pk, pv, ps, pq) in enumerate(pools)]
        sfn = lambda i: steps_[i % copies]()  # noqa: E731
        for i in range(200):
            sfn(i)
        step = {"step_us": round(back_to_back_us(torch, sfn, calls), 2),
                "step_per_call_us": pct(timed_calls(torch, sfn, calls)),
                "step_launches": 1 if band_sizes[1] >= 1 else (3 if sq else 2)}
        del steps_
    res = {"workload": case_label(name, layer, key_scale, band_sizes, fp8, sq, wl),
           "batch": B, "seq_len": S, "q_heads": Hq, "kv_heads": H, "head_dim": D,
           "paged_block": wl.block_size or None, "code_bytes": cb, "scale_bytes": sb,
           "band_bytes": bb, "pool_copies": copies, "pool_bytes_rotated": pool_bytes * copies,
           "band_copies": band_copies if band_sizes else None,
           "decode_us": round(us, 2), "per_call_us": pct(per_call),
           "GB_per_s": round((cb + sb + bb) / (us * 1e-6) / 1e9, 1),
           "frac_of_hbm_peak": round((cb + sb + bb) / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4), **step}
    del pools, calls_, ws, bands
    torch.cuda.empty_cache()
    return res


def append_encode(nk, torch, dev, P, gen):
    """Prefill-encode of 4096 new tokens x 32 sequences x 8 KV heads into a paged
    cache of 16-token blocks with a shuffled block table."""
    import synth
    awl = synth.get_workload("append_paged")
    H, D, L = awl.num_kv_heads, awl.head_dim, awl.groups
    kk = torch.randn((awl.batch, awl.n_new, H, D), generator=gen, device=dev).to(torch.bfloat16)
    vv = torch.randn((awl.batch, awl.n_new, H, D), generator=gen, device=dev).to(torch.bfloat16)
    bps = awl.seq_len // awl.block_size
    table = torch.as_tensor(synth.shuffled_block_table(awl)).to(dev)
    alay = nk.CacheLayout(awl.block_size, bps, table)
    apk = torch.zeros((awl.batch * bps, H, awl.block_size, L), dtype=torch.uint8, device=dev)
    apv = torch.zeros_like(apk)
    sp = torch.full((awl.batch,), awl.seq_len - awl.n_new, dtype=torch.int32, device=dev)
    call = nk.prepare_encode(P, alay, kk, vv, sp, apk, apv)
    call()
    per_call = timed_calls(torch, lambda i: call(), 10)
    a_ms = float(np.median(per_call)) * 1e-3
    th = awl.batch * awl.n_new * H
    flops = th * ENCODE_FLOPS_PER_TOKEN_HEAD
    tflops = flops / (a_ms * 1e-3) / 1e12
    return {"workload": "append 4096 tokens x 32 sequences, 8 KV heads, D=128, paged 16-token blocks",
            "ms": round(a_ms, 3), "per_call_us": pct(per_call),
            "token_heads_per_s": round(th / (a_ms * 1e-3), 1),
            "roofline": {"bound": "mfma", "dtype": "f64", "achieved": round(tflops, 2),
                         "peak": FP64_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(tflops / FP64_MFMA_PEAK_TFLOPS, 4),
                         "algorithmic_flops": flops,
                         "flops_per_token_head": ENCODE_FLOPS_PER_TOKEN_HEAD}}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(the decode shards by KV head with no exchange; see the design notes).",
              file=sys.stderr)
        sys.exit(2)

    # the oracle on the host cores first, before anything touches the GPU
    cpu = None
    if not args.no_cpu_baseline and args.only is None:
        cpu = cpu_baseline(args.cpu_seconds)
        print(f"[bench] cpu baseline done: {cpu['us_per_step']} us per step on {cpu['cores']} cores",
              file=sys.stderr, flush=True)

    import torch

    import paper_2608_04074_amd as nk
    import synth

    wl = synth.get_workload(WORKLOAD)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B, S, H, Hq, D, L = wl.batch, wl.seq_len, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.groups
    code_bytes = wl.code_bytes_per_step()
    gen = torch.Generator(device=dev)
    gen.manual_seed(1234)
    params = synth.bench_params(wl)
    P = nk.NovaKVParams.from_arrays(params, device=dev)

    if args.only is not None:
        if args.only == "append_encode":
            line = append_encode(nk, torch, dev, P, gen)
        else:
            import synth as _s
            case = next((c for c in OTHER_CASES
                         if case_label(*c, _s.get_workload(c[0])).startswith(args.only)), None)
            if case is None:
                print(f"no workload line starts with {args.only!r}", file=sys.stderr)
                sys.exit(2)
            line = other_workload(nk, torch, dev, case, args.calls)
        if args.copy_calib:
            copy_calibration(torch, dev)
        print(json.dumps({"only": args.only, "line": line}), flush=True)
        return

    # the other workload shapes and the append encoder (reported beside the headline)
    others = None
    if not args.skip_others:
        others = []
        for case in OTHER_CASES:
            others.append(other_workload(nk, torch, dev, case, args.calls))
            print(f"[bench] {others[-1]['workload']}: {others[-1]['decode_us']} us", file=sys.stderr, flush=True)
    append = None if args.skip_append else append_encode(nk, torch, dev, P, gen)

    # ---- the headline step
    layout = nk.CacheLayout.contiguous(S)
    copies = rotation_copies(2 * B * H * S * L, at_least=6)
    pools = [(torch.randint(0, 256, (B, H, S, L), dtype=torch.uint8, device=dev, generator=gen),
              torch.randint(0, 256, (B, H, S, L), dtype=torch.uint8, device=dev, generator=gen))
             for _ in range(copies)]
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
        step_calls[i % copies]()

    def two_call_step(i):
        enc_calls[i % copies]()
        dec_calls[i % copies]()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    # the timed region: exactly `steps` steps, synchronized on both sides
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for i in range(args.steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_step = e0.elapsed_time(e1) / args.steps

    # beside the timed region: per-call distributions and the parts of the step
    n_pc = max(200, args.steps)
    step_pc = timed_calls(torch, step, n_pc)
    two_call_us = back_to_back_us(torch, two_call_step, n_pc)
    dec_us = back_to_back_us(torch, lambda i: dec_calls[i % copies](), n_pc)
    dec_pc = timed_calls(torch, lambda i: dec_calls[i % copies](), n_pc)
    enc_us = back_to_back_us(torch, lambda i: enc_calls[i % copies](), n_pc)
    # the same step with the codebooks in the paper's stored format: rounded to
    # fp8 E4M3 (torch's conversion) and passed as bytes
    p8 = dict(params)
    for k in ("cb_k", "cb_v"):
        p8[k] = torch.as_tensor(params[k]).to(torch.float32).to(torch.float8_e4m3fn).view(torch.uint8)
    P8 = nk.NovaKVParams.from_arrays(p8, device=dev)
    step8_calls = [nk.prepare_append_decode(P8, layout, k_new[:, 0], v_new[:, 0], q, pk, pv, seq_lens, S, out, ws)
                   for pk, pv in pools]
    for i in range(200):
        step8_calls[i % copies]()
    step8_us = back_to_back_us(torch, lambda i: step8_calls[i % copies](), n_pc)
    # the paper's serving storage: these codebooks in fp8 and the bases
    # (t_k, t_k_inv_t, t_v) in bf16
    PS = nk.NovaKVParams.from_arrays(p8, device=dev, bf16_transforms=True)
    steps_calls = [nk.prepare_append_decode(PS, layout, k_new[:, 0], v_new[:, 0], q, pk, pv, seq_lens, S, out, ws)
                   for pk, pv in pools]
    for i in range(200):
        steps_calls[i % copies]()
    step_serving_us = back_to_back_us(torch, lambda i: steps_calls[i % copies](), n_pc)

    if args.copy_calib:  # plain copy of known size, last dispatch of the run
        copy_calibration(torch, dev)

    value = code_bytes / (ms_step * 1e-3) / 1e9
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
        "dtype": "f16-mfma-f32acc",
        "data": "synthetic",
        "config": {
            "workload": "qwen3_8b-shaped GQA decode layer over a 2-bit VQ K/V cache: encode 1 new token "
                        "per sequence + decode attention, one launch",
            "batch": B, "seq_len": S, "q_heads": Hq, "kv_heads": H, "head_dim": D,
            "code_bytes_per_step": code_bytes, "pool_copies": copies,
            "params": "random orthogonal transforms, fp16 N(0,1) codebooks, uniform random codes",
            "arithmetic": "fp16 table entries and probabilities on MFMA with fp32 accumulation; fp32 softmax, "
                          "query transform and combine; fp64 encoder",
        },
        "timed_region_wall_s": round(t_wall, 4),
        "step_per_call_us": pct(step_pc),
        "step_fp8_codebooks_us": round(step8_us, 2),
        "step_bf16_bases_fp8_codebooks_us": round(step_serving_us, 2),
        "two_call_step_us": round(two_call_us, 2),
        "decode_kernel_us": {"mean": round(dec_us, 2), **pct(dec_pc)},
        "append_kernel_us": round(enc_us, 2),
        "roofline": {
            "kernel": f"{DECODE_KERNEL}<12, true, false, false, false, false, false> (the step's one launch: encode of the new token, query "
                      "transform, split pass, combine)",
            "bound": "hbm",
            "achieved": round(value, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(value / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "counters": measured_counters(),
            "algorithmic_bytes_per_launch": code_bytes,
            "algorithmic_bytes_per_token_head": 2 * L,
        },
        "append_encode": append,
        "other_workloads_decode": others,
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


def copy_calibration(torch, dev):
    src = torch.empty(COPY_CALIB_BYTES, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()


if __name__ == "__main__":
    main()
