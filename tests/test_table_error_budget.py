"""Error budget of the table kernels' arithmetic, on the CPU.

A model of the roundings the decode kernels make, against the fp64 oracle:
the query transform in fp32, the table of partial logits built from the
query split into two fp16 halves and rounded to fp16, logits summed in fp32
(log2 units), probabilities rounded to fp16 for the value product, fp32
denominators, accumulators and inverse value transform.  Over workload-shaped
heads (the synthetic GPT-OSS-20B and Qwen3-8B queries and calibrations,
uniformly random codes, sinks where the workload has them) it measures the
row error the parity tests bound by 2e-3, and which rounding dominates it.
"""

import numpy as np
import pytest

import synth
from helpers import TOL, row_errors
from oracle import attention as oatt
from oracle_cache import calibrated_params

LOG2E = 1.4426950408889634
f16, f32 = np.float16, np.float32


def table_path_rows(q, ck, cv, hp, scale, sinks=None, table_fp16=True, probs_fp16=True):
    """Outputs (G, D) of the G query heads of one KV head under the kernels' roundings."""
    G, D = q.shape
    L = D // 4
    qp = (q.astype(f32) @ np.asarray(hp["t_k_inv_t"], f32)) * f32(scale * LOG2E)
    hi = qp.astype(f16)
    lo = (qp - hi.astype(f32)).astype(f16)
    cb = np.asarray(hp["cb_k"], f16).astype(f32)                      # (L, 256, 4)
    table = (np.einsum("glj,lcj->lcg", hi.astype(f32).reshape(G, L, 4), cb).astype(f32)
             + np.einsum("glj,lcj->lcg", lo.astype(f32).reshape(G, L, 4), cb).astype(f32))
    if table_fp16:
        table = table.astype(f16).astype(f32)
    z = np.zeros((ck.shape[0], G), f32)
    for g in range(L):
        z += table[g, ck[:, g], :]
    m = z.max(axis=0)
    p = np.exp2(z - m).astype(f32)
    den = p.sum(axis=0, dtype=f32)
    cv_tab = np.asarray(hp["cb_v"], f16).astype(f32)
    s_hat = np.stack([cv_tab[g, cv[:, g], :] for g in range(L)], axis=1).reshape(ck.shape[0], D)
    acc = (p.astype(f16).astype(f32) if probs_fp16 else p).T @ s_hat
    if sinks is not None:  # the sink, shifted by -(q . k_bar) * scale, in natural-log units
        shift = np.asarray(sinks, f32) - f32(scale) * (q.astype(f32) @ np.asarray(hp["kbar"], f32))
        den = den + np.exp(shift - m * f32(np.log(2.0))).astype(f32)
    return ((acc / den[:, None]) @ np.asarray(hp["t_v"], f32).T).astype(np.float64)


def _errors(name, layer, lengths, batch, **kw):
    wl = synth.get_workload(name)
    G, D, L = wl.gqa, wl.head_dim, wl.groups
    params = calibrated_params(wl, layer)
    queries = synth.decode_queries(wl, layer, batch=batch)
    sinks_all = synth.sink_logits(wl, layer)
    rng = np.random.default_rng(100 + layer)
    out = []
    for S in lengths:
        for b in range(batch):
            for kv in range(wl.num_kv_heads):
                hp = oatt.head_params(params, kv)
                ck = rng.integers(0, 256, (S, L))
                cv = rng.integers(0, 256, (S, L))
                q = queries[b, kv * G:(kv + 1) * G]
                sinks = None if sinks_all is None else sinks_all[kv * G:(kv + 1) * G]
                ref = oatt.decode_rows(q, ck, cv, hp, 1 / np.sqrt(D), 0, sinks)
                out.append(row_errors(table_path_rows(q, ck, cv, hp, 1 / np.sqrt(D), sinks, **kw), ref))
    return np.concatenate(out)


@pytest.mark.parametrize("name,layer,bound", [("gptoss_pair", 0, 0.9 * TOL), ("gptoss_pair", 1, 0.9 * TOL),
                                              ("qwen3_8b", 0, 0.5 * TOL)])
def test_table_arithmetic_stays_inside_the_tolerance(name, layer, bound):
    """Over 2048+ workload-shaped rows the modelled kernel error stays below
    the bound; the D=64 shape (eight query heads, larger logits) has the
    smaller margin."""
    e = _errors(name, layer, [1, 3, 16, 128, 700], 8)
    print(f"[budget] {name} L{layer}: rows={e.size} median={np.median(e):.2e} "
          f"p99={np.percentile(e, 99):.2e} max={e.max():.2e} tol={TOL}")
    assert e.max() <= bound


def test_table_rounding_dominates_the_error():
    """The worst rows come from the fp16 partial-logit table: with an fp32
    table their error drops several-fold, with fp32 probabilities it barely
    moves (the probabilities' rounding matters only in the typical rows)."""
    full = _errors("gptoss_pair", 1, [16, 128, 700], 4)
    t32 = _errors("gptoss_pair", 1, [16, 128, 700], 4, table_fp16=False)
    p32 = _errors("gptoss_pair", 1, [16, 128, 700], 4, probs_fp16=False)
    q = lambda e: np.percentile(e, 99.5)  # noqa: E731
    print(f"[budget] p99.5 full={q(full):.2e} fp32 table={q(t32):.2e} fp32 probabilities={q(p32):.2e}")
    assert q(t32) * 3 < q(full)
    assert q(p32) > 0.7 * q(full)
