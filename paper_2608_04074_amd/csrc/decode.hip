// Decode attention over the 2-bit VQ cache: query pre-transform, split-context
// stage 1 (codebook gather, online softmax, transform-domain value
// accumulation) and split combine with one inverse value transform per head.
//
// Paper: Algorithm 1 (attention step), Sec. "Decoding kernel and read path"
// (q R_K^{-T} once per step, per-group codeword lookup, k_bar dropped by
// Lemma S1, two-stage split-KV decode), Corollary 1 (v_hat = s_hat R_V^T) and
// the sinks appendix (sink added once after the combine, shifted by
// -(q . k_bar) * scale).
#include <math.h>

#include "nova_kv_internal.h"

namespace novakv {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// q'[b][h] = (q[b][h] @ t_k_inv_t[kv]) * scale and the shifted sink logit.
template <int D>
__global__ void __launch_bounds__(D) decode_prologue(DecodeArgs a) {
  const int bh = blockIdx.x;
  const int h = bh % a.num_q_heads;
  const int kv = h / a.gqa;
  const int tid = threadIdx.x;
  __shared__ float qsh[D];
  __shared__ float red[D / 64];
  float qv;
  if (a.q_bf16)
    qv = bf16_bits_to_float(static_cast<const uint16_t *>(a.q)[static_cast<size_t>(bh) * D + tid]);
  else
    qv = static_cast<const float *>(a.q)[static_cast<size_t>(bh) * D + tid];
  qsh[tid] = qv;
  float dotk = wave_sum(qv * a.kbar[kv * D + tid]);
  if ((tid & 63) == 0) red[tid >> 6] = dotk;
  __syncthreads();
  const void *tk = transform_of(a.t_k_inv_t, kv, D, a.t_bf16);
  float acc = 0.f;
#pragma unroll 16
  for (int d = 0; d < D; ++d) acc = fmaf(qsh[d], t1_value(tk, static_cast<size_t>(d) * D + tid, a.t_bf16), acc);
  a.qp[static_cast<size_t>(bh) * D + tid] = acc * a.qscale;
  if (tid == 0) {
    float s = 0.f;
    for (int w = 0; w < D / 64; ++w) s += red[w];
    a.sinkp[bh] = a.sinks ? a.sinks[h] - s * a.scale : -INFINITY;
  }
}

// Stage 1: one workgroup per (split, KV head, sequence); one token per thread
// for the scores, one transform-domain coordinate per thread for the values.
template <int D>
__global__ void __launch_bounds__(kThreads) decode_stage1_v0(DecodeArgs a) {
  constexpr int L = D / kGroupDim;
  constexpr int CB = L * kCodebookSize * kGroupDim;  // halves per side
  __shared__ __attribute__((aligned(16))) uint16_t cbk[CB];
  __shared__ __attribute__((aligned(16))) uint16_t cbv[CB];
  __shared__ float qs[kMaxGqa][D];
  __shared__ float ps[kThreads][kMaxGqa];
  __shared__ __attribute__((aligned(16))) uint8_t vcodes[kThreads][L];
  __shared__ float vsq[kThreads][2];  // scalar value arm: scale, offset of each token
  __shared__ float red[kWaves][kMaxGqa];

  const int split = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int G = a.gqa;

  // the pools are read for [lo, tend): the attended span without the band
  const int S = a.seq_lens[b];
  const AttendedSpans spn = attended_spans(a.window > 0 ? max(0, S - a.window) : 0, S, a.n_sink, a.n_rec);
  const int lo = spn.code_lo, tend = spn.code_hi;
  {  // a split beyond that span publishes an empty partial and stops
    if (lo + split * a.chunk >= tend) {
      const size_t row0 = static_cast<size_t>(b) * a.num_q_heads + kv * G;
      for (int i = tid; i < G * D; i += kThreads) {
        const size_t r = (row0 + i / D) * a.n_split + split;
        a.part_acc[r * D + i % D] = 0.f;
        if (i % D == 0) {
          a.part_ml[2 * r] = -INFINITY;
          a.part_ml[2 * r + 1] = 0.f;
        }
      }
      return;
    }
  }

  {
    // both codebooks into LDS as fp16 (fp8 codewords converted on the way)
    const size_t cw0 = static_cast<size_t>(kv) * L * kCodebookSize;
    uint2 *dk = reinterpret_cast<uint2 *>(cbk);
    uint2 *dv = reinterpret_cast<uint2 *>(cbv);
    for (int i = tid; i < L * kCodebookSize; i += kThreads) {
      dk[i] = codeword(a.cb_k, a.cb_fp8, cw0 + i);
      if (!a.v_sq) dv[i] = codeword(a.cb_v, a.cb_fp8, cw0 + i);
    }
    for (int i = tid; i < G * D; i += kThreads)
      qs[i / D][i % D] =
          a.qp[(static_cast<size_t>(b) * a.num_q_heads + kv * G + i / D) * D + (i % D)];
  }

  const int t0 = lo + split * a.chunk;  // splits tile the span [lo, tend)
  const int t1 = min(tend, lo + (split + 1) * a.chunk);

  float m[kMaxGqa], l[kMaxGqa], acc[kMaxGqa];
#pragma unroll
  for (int h = 0; h < kMaxGqa; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.f;
    acc[h] = 0.f;
  }
  __syncthreads();

  const int wave = tid >> 6, lane = tid & 63;
  for (int ts = t0; ts < t1; ts += kThreads) {
    const int t = ts + tid;
    const bool valid = t < t1;
    float z[kMaxGqa];
#pragma unroll
    for (int h = 0; h < kMaxGqa; ++h) z[h] = valid ? 0.f : -INFINITY;
    if (valid) {
      const size_t off = code_row_offset(a.layout, a.num_kv_heads, L, b, kv, t);
      const uint8_t *kc = a.k_codes + off;
      const uint8_t *vc = a.v_codes + off;
      if (a.v_sq) {
        vsq[tid][0] = bf16_bits_to_float(a.v_sq[(off / L) * 2]);
        vsq[tid][1] = bf16_bits_to_float(a.v_sq[(off / L) * 2 + 1]);
      }
      for (int g0 = 0; g0 < L; g0 += 16) {
        uint4 w = *reinterpret_cast<const uint4 *>(kc + g0);
        *reinterpret_cast<uint4 *>(&vcodes[tid][g0]) = *reinterpret_cast<const uint4 *>(vc + g0);
        const uint32_t words[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int ell = g0 + j;
          const int c = (words[j >> 2] >> (8 * (j & 3))) & 0xff;
          const uint16_t *cw = &cbk[(ell * kCodebookSize + c) * kGroupDim];
          const float f0 = half_bits_to_float(cw[0]);
          const float f1 = half_bits_to_float(cw[1]);
          const float f2 = half_bits_to_float(cw[2]);
          const float f3 = half_bits_to_float(cw[3]);
#pragma unroll
          for (int h = 0; h < kMaxGqa; ++h) {
            if (h < G) {
              const float *qh = &qs[h][ell * kGroupDim];
              z[h] = fmaf(qh[0], f0, fmaf(qh[1], f1, fmaf(qh[2], f2, fmaf(qh[3], f3, z[h]))));
            }
          }
        }
      }
      if (a.k_scales) {  // key-scale format: the read path's per-token multiply
        const float rho = __uint_as_float(static_cast<uint32_t>(a.k_scales[off / L]) << 16);
#pragma unroll
        for (int h = 0; h < kMaxGqa; ++h) z[h] *= rho;
      }
    }
    // tile max per head
#pragma unroll
    for (int h = 0; h < kMaxGqa; ++h) {
      if (h < G) {
        const float wm = wave_max(z[h]);
        if (lane == 0) red[wave][h] = wm;
      }
    }
    __syncthreads();
    float mnew[kMaxGqa], alpha[kMaxGqa];
#pragma unroll
    for (int h = 0; h < kMaxGqa; ++h) {
      if (h < G) {
        float tm = red[0][h];
        for (int w = 1; w < kWaves; ++w) tm = fmaxf(tm, red[w][h]);
        mnew[h] = fmaxf(m[h], tm);
        alpha[h] = (m[h] == -INFINITY) ? 0.f : __expf(m[h] - mnew[h]);
        ps[tid][h] = valid ? __expf(z[h] - mnew[h]) : 0.f;
      }
    }
    __syncthreads();  // red reused below; ps and vcodes complete
#pragma unroll
    for (int h = 0; h < kMaxGqa; ++h) {
      if (h < G) {
        const float ws = wave_sum(ps[tid][h]);
        if (lane == 0) red[wave][h] = ws;
      }
    }
    if (tid < D) {
      const int ell = tid >> 2, i = tid & 3;
      const int n = min(kThreads, t1 - ts);
#pragma unroll
      for (int h = 0; h < kMaxGqa; ++h) acc[h] *= (h < G) ? alpha[h] : 0.f;
      for (int j = 0; j < n; ++j) {
        const int c = vcodes[j][ell];
        // a codeword coordinate, or the scalar arm's offset + scale * q
        const float f = a.v_sq ? fmaf(vsq[j][0], static_cast<float>((c >> (2 * i)) & 3), vsq[j][1])
                               : half_bits_to_float(cbv[(ell * kCodebookSize + c) * kGroupDim + i]);
#pragma unroll
        for (int h = 0; h < kMaxGqa; ++h)
          if (h < G) acc[h] = fmaf(ps[j][h], f, acc[h]);
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < kMaxGqa; ++h) {
      if (h < G) {
        float tsum = 0.f;
        for (int w = 0; w < kWaves; ++w) tsum += red[w][h];
        l[h] = l[h] * alpha[h] + tsum;
        m[h] = mnew[h];
      }
    }
    __syncthreads();  // red and ps free for the next tile
  }

  const size_t row0 = static_cast<size_t>(b) * a.num_q_heads + kv * G;
  for (int h = 0; h < G; ++h) {
    const size_t r = (row0 + h) * a.n_split + split;
    if (tid < D) a.part_acc[r * D + tid] = acc[h];
    if (tid == 0) {
      a.part_ml[2 * r] = m[h];
      a.part_ml[2 * r + 1] = l[h];
    }
  }
}

// Stage 2, one workgroup per (sequence, KV head): log-sum-exp merge of the
// splits, sink once, the sink-plus-recent band (when there is one) as one
// more partial, divide, then v = s t_v^T for the KV head's query heads (t_v
// read once per workgroup, rows as 16-byte vectors) plus the band's value
// term, which is in the original domain.
//
// Band (paper: Sec. "Sink-plus-recent band"): positions [lo, sink_end) and
// [code_hi, S) with their bf16 keys and values; logits
// z = (q . k - q . k_bar) * scale, the shift of the codes' logits (Lemma S1).
template <int D>
__global__ void __launch_bounds__(256) decode_combine(DecodeArgs a) {
  const int b = blockIdx.x / a.num_kv_heads;
  const int kv = blockIdx.x - b * a.num_kv_heads;
  const int G = a.gqa;
  const int tid = threadIdx.x;
  __shared__ float sh[kMaxGqa][D];
  __shared__ float bq[kMaxGqa][D];           // band: query, later the value sums
  __shared__ float bz[kMaxBand][kMaxGqa];    // band logits, then probabilities
  __shared__ float bpart[256 / D][kMaxGqa][D];
  __shared__ float bst[3][kMaxGqa];          // q . k_bar, max, sum
  __shared__ float bout[kMaxGqa][D];
  const int S = a.seq_lens[b];
  const int att_lo = a.window > 0 ? max(0, S - a.window) : 0;
  const AttendedSpans spn = attended_spans(att_lo, S, a.n_sink, a.n_rec);
  const int ns = max(0, spn.sink_end - att_lo);
  const int nband = a.band_k ? ns + (S - spn.code_hi) : 0;
  if (nband > 0) {
    const size_t hb = (static_cast<size_t>(b) * a.num_kv_heads + kv) * (a.n_sink + a.n_rec);
    auto row_of = [&](const int i) -> size_t {
      const int p = i < ns ? att_lo + i : spn.code_hi + (i - ns);
      return (hb + band_slot(p, a.n_sink, a.n_rec)) * D;
    };
    for (int i = tid; i < G * D; i += 256) {
      const size_t qi = (static_cast<size_t>(b) * a.num_q_heads + kv * G) * D + i;
      bq[i / D][i % D] = a.q_bf16 ? bf16_bits_to_float(static_cast<const uint16_t *>(a.q)[qi])
                                  : static_cast<const float *>(a.q)[qi];
    }
    __syncthreads();
    if (tid < G) {
      float x = 0.f;
      for (int d = 0; d < D; ++d) x = fmaf(bq[tid][d], a.kbar[kv * D + d], x);
      bst[0][tid] = x;
    }
    __syncthreads();
    for (int i = tid; i < nband; i += 256) {  // one band row per thread
      const uint4 *kr = reinterpret_cast<const uint4 *>(a.band_k + row_of(i));
      float z[kMaxGqa];
#pragma unroll
      for (int h = 0; h < kMaxGqa; ++h) z[h] = 0.f;
      for (int c = 0; c < D / 8; ++c) {
        const uint4 w = kr[c];
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float kx = __uint_as_float((e & 1) ? (ws[e >> 1] & 0xffff0000u) : (ws[e >> 1] << 16));
#pragma unroll
          for (int h = 0; h < kMaxGqa; ++h)
            if (h < G) z[h] = fmaf(bq[h][8 * c + e], kx, z[h]);
        }
      }
#pragma unroll
      for (int h = 0; h < kMaxGqa; ++h)
        if (h < G) bz[i][h] = (z[h] - bst[0][h]) * a.scale;
    }
    __syncthreads();
    for (int h = tid >> 6; h < G; h += 4) {  // one wave per head
      const int lane = tid & 63;
      float mx = -INFINITY;
      for (int i = lane; i < nband; i += 64) mx = fmaxf(mx, bz[i][h]);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
      float l = 0.f;
      for (int i = lane; i < nband; i += 64) {
        const float p = __expf(bz[i][h] - mx);
        bz[i][h] = p;
        l += p;
      }
      l = wave_sum(l);
      if (lane == 0) {
        bst[1][h] = mx;
        bst[2][h] = l;
      }
    }
    __syncthreads();
    {  // values: thread (part, d) takes rows i = part mod 256 / D
      constexpr int PARTS = 256 / D;
      const int d = tid % D, part = tid / D;
      float acc[kMaxGqa];
#pragma unroll
      for (int h = 0; h < kMaxGqa; ++h) acc[h] = 0.f;
      for (int i = part; i < nband; i += PARTS) {
        const float v = bf16_bits_to_float(a.band_v[row_of(i) + d]);
#pragma unroll
        for (int h = 0; h < kMaxGqa; ++h)
          if (h < G) acc[h] = fmaf(bz[i][h], v, acc[h]);
      }
#pragma unroll
      for (int h = 0; h < kMaxGqa; ++h) bpart[part][h][d] = acc[h];
    }
    __syncthreads();
    for (int i = tid; i < G * D; i += 256) {
      float x = 0.f;
      for (int p = 0; p < 256 / D; ++p) x += bpart[p][i / D][i % D];
      bq[i / D][i % D] = x;
    }
    __syncthreads();
  }
  for (int i = tid; i < G * D; i += 256) {
    const int h = i / D, d = i - h * D;
    const size_t bh = static_cast<size_t>(b) * a.num_q_heads + kv * G + h;
    const float *ml = a.part_ml + bh * a.n_split * 2;
    const float *pa = a.part_acc + bh * a.n_split * D;
    const float sink = a.sinkp[bh];
    float big = sink;
    for (int s = 0; s < a.n_split; ++s) big = fmaxf(big, ml[2 * s]);
    float den = 0.f, num = 0.f;
    if (big != -INFINITY) {
      for (int s = 0; s < a.n_split; ++s) {
        const float ms = ml[2 * s];
        const float w = (ms == -INFINITY) ? 0.f : __expf(ms - big);
        den = fmaf(w, ml[2 * s + 1], den);
        num = fmaf(w, pa[static_cast<size_t>(s) * D + d], num);
      }
      if (sink != -INFINITY) den += __expf(sink - big);
    }
    float bo = 0.f;
    if (nband > 0) {  // the band after the splits and the sink
      const float mb = bst[1][h];
      if (mb > big) {
        const float f = big == -INFINITY ? 0.f : __expf(big - mb);
        num *= f;
        den *= f;
        big = mb;
      }
      const float wb = __expf(mb - big);
      den = fmaf(wb, bst[2][h], den);
      bo = wb * bq[h][d];
    }
    sh[h][d] = (den > 0.f) ? num / den : 0.f;
    bout[h][d] = (den > 0.f) ? bo / den : 0.f;
  }
  __syncthreads();
  // thread -> (output coordinate d, half of the heads)
  constexpr int HALVES = 256 / D;
  const int d = tid % D, part = tid / D;
  const void *tv = transform_of(a.t_v, kv, D, a.t_bf16);
  float o[kMaxGqa];
#pragma unroll
  for (int h = 0; h < kMaxGqa; ++h) o[h] = 0.f;
#pragma unroll 8
  for (int j4 = 0; j4 < D / 4; ++j4) {
    const float4 w = t4_value(load_t4(tv, static_cast<size_t>(d) * D + 4 * j4, a.t_bf16), a.t_bf16);
#pragma unroll
    for (int h = 0; h < kMaxGqa; ++h) {
      if (h % HALVES == part && h < G) {
        o[h] = fmaf(sh[h][4 * j4 + 0], w.x, o[h]);
        o[h] = fmaf(sh[h][4 * j4 + 1], w.y, o[h]);
        o[h] = fmaf(sh[h][4 * j4 + 2], w.z, o[h]);
        o[h] = fmaf(sh[h][4 * j4 + 3], w.w, o[h]);
      }
    }
  }
#pragma unroll
  for (int h = 0; h < kMaxGqa; ++h)
    if (h % HALVES == part && h < G)
      a.out[(static_cast<size_t>(b) * a.num_q_heads + kv * G + h) * D + d] = nband > 0 ? o[h] + bout[h][d] : o[h];
}

template <int D>
hipError_t launch_decode_d(const DecodeArgs &a, int use_lut, hipStream_t stream) {
  if (use_lut) return D == 128 ? launch_decode_lut(a, stream) : launch_decode_lut64(a, stream);
  const int rows = a.batch * a.num_q_heads;
  decode_prologue<D><<<dim3(rows), dim3(D), 0, stream>>>(a);
  decode_stage1_v0<D><<<dim3(a.n_split, a.num_kv_heads, a.batch), dim3(kThreads), 0, stream>>>(a);
  decode_combine<D><<<dim3(a.batch * a.num_kv_heads), dim3(256), 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace

namespace {

void plan_generic(int batch, int num_kv_heads, int max_seq_len, int *n_split, int *chunk) {
  int c = 1024;
  auto splits = [&](int cc) { return (max_seq_len + cc - 1) / cc; };
  while (c > 64 && static_cast<long long>(batch) * num_kv_heads * splits(c) < 2048) c /= 2;
  *chunk = c;
  *n_split = splits(c);
}

}  // namespace

DecodePlan plan_decode(int batch, int num_q_heads, int num_kv_heads, int head_dim,
                       int max_seq_len, int block_size, int window, bool split_k_only) {
  DecodePlan p{};
  const int gqa = num_q_heads / num_kv_heads;
  // Splits tile the attended span: the last `window` tokens, or all of them.
  const int span = window > 0 && window < max_seq_len ? window : max_seq_len;
  int ns_g, ch_g, ns_l, ch_l;
  plan_generic(batch, num_kv_heads, max_seq_len, &ns_g, &ch_g);
  ns_g = (span + ch_g - 1) / ch_g;  // the full-context chunk, so a window never adds splits
  plan_lut(batch, num_kv_heads, span, &ns_l, &ch_l);
  // Workspace bound over every window: the full-context generic plan, and the
  // table plan's split target (its split count never exceeds it).
  int ns_full, ch_full;
  plan_generic(batch, num_kv_heads, max_seq_len, &ns_full, &ch_full);
  const long long units = static_cast<long long>(batch) * num_kv_heads;
  const int lut_bound = static_cast<int>((256 + units - 1) / units);
  int max_split = ns_full > lut_bound ? ns_full : lut_bound;
  if (block_size > 0) {
    p.use_lut = !split_k_only && lut_path_eligible(head_dim, gqa, block_size) ? 1 : 0;
    p.n_split = p.use_lut ? ns_l : ns_g;
    p.chunk = p.use_lut ? ch_l : ch_g;
  } else {
    p.use_lut = 0;
    p.n_split = ns_g;
    p.chunk = ch_g;
  }
  if (p.n_split > max_split) max_split = p.n_split;
  auto align = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
  const size_t rows = static_cast<size_t>(batch) * num_q_heads;
  // groups of the two-level combine, at most, over every split count up to the bound
  int max_group = 1;
  for (int n = 1; n <= max_split; ++n) {
    const int gs = plan_group_size(n), ng = (n + gs - 1) / gs;
    if (ng > max_group) max_group = ng;
  }
  p.off_cnt = 0;
  p.off_qp = align(static_cast<size_t>(units) * (1 + max_group) * sizeof(int));
  p.off_sinkp = align(p.off_qp + rows * head_dim * sizeof(float));
  p.off_ml = align(p.off_sinkp + rows * sizeof(float));
  p.off_acc = align(p.off_ml + rows * max_split * 2 * sizeof(float));
  p.off_new = align(p.off_acc + rows * max_split * head_dim * sizeof(float));
  p.off_xch = align(p.off_new + static_cast<size_t>(batch) * num_kv_heads * 8 * 32 * sizeof(float));
  p.off_xnew = align(p.off_xch + units * max_split * kXchSlotWords * sizeof(uint64_t));
  p.off_xgrp = align(p.off_xnew + static_cast<size_t>(units) * 8 * 32 * sizeof(uint64_t));
  p.total = align(p.off_xgrp + units * max_group * kXchSlotWords * sizeof(uint64_t));
  return p;
}

hipError_t launch_decode(const DecodeArgs &a, int use_lut, hipStream_t stream) {
  switch (a.head_dim) {
    case 64: return launch_decode_d<64>(a, use_lut, stream);
    case 128: return launch_decode_d<128>(a, use_lut, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace novakv
