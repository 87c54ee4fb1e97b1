// Decode attention for head_dim 64 and up to 8 query heads per KV head (the
// GPT-OSS-20B shape), in one launch.  Same method as the head_dim-128 table
// kernel: per-query table of partial logits, transposing LDS gathers summed on
// the matrix cores, per-column online softmax, values accumulated in the
// transform domain, and the split combine by the last arriving split.
//
// Paper: Algorithm 1 (attention step); Theorem 1 (q' = q R_K^{-T}); Sec.
// "Decoding kernel and read path" (query transformed once per step, one
// codebook lookup per group, k_bar dropped by Lemma S1, split-KV decode);
// Corollary 1 (v_hat = s_hat R_V^T); appendix on attention sinks.
//
// Differences from the head_dim-128 kernel:
//  * 16 groups, 8 heads per table entry: LUT[c][g][h] (fp16, 16 B) at
//    c*256 + g*16 + 8*(h/4); a transposing read fetches one half (4 heads).
//  * A round is 64 tokens in two halves of 32, whose key work, then softmax,
//    then value work are issued together.  Within a half, read lane
//    (rho, j, tq, hh) = 16 rho + 4 j + 2 tq + hh gathers half hh of group
//    4j + ((2(rho&1) + tq) ^ t) of token 8r + 2 rho + tq at step t: a half-wave
//    touches 16 groups x 2 halves, i.e. 32 distinct bank pairs.  The selector
//    MFMA leaves lane (tau, set, head) = 16 tau + 8 set + head with the logits
//    of tokens 8 tau + 2 i + set of the half.
//  * Values: two token sets per half, 4 coordinate tiles of 16.
#include <math.h>

#include "band_attention.h"
#include "lut_common.h"
#include "nova_kv_internal.h"
#include "step_encode.h"

namespace novakv {

namespace {

using namespace lut;

constexpr int kD = 64;
constexpr int kL = kD / kGroupDim;     // 16 groups
constexpr int kH = 8;                  // heads per table entry
constexpr int kRound = 64;             // tokens per round: two halves of 32
constexpr int kBuf = 2;                // rounds of code bytes in flight per wave
constexpr uint32_t kLutBytes = 65536;  // [256 codes][16 groups][8 heads] fp16
constexpr uint32_t kVBase = kLutBytes; // value codebook, 32 KB
constexpr uint32_t kMergeBase = 0;     // per-wave merge scratch, reuses the table once done
constexpr int kMergeFloats = kH * kD + 2 * kH;
constexpr float kLazyLog2 = 8.f;       // reference lag allowed in the online softmax (log2 units)
// Auxiliary region: query staging, partial sums of q' (4 parts), later the
// split's own partial ([8][64]) and the combine's partial outputs ([4][8][64]).
constexpr uint32_t kAuxQ = kVBase + 32768;          // [8][64] f32
constexpr uint32_t kAuxPart = kAuxQ + kH * kD * 4;  // 10 KB
constexpr uint32_t kAuxOwn = kAuxPart;
constexpr uint32_t kAuxOut = kAuxPart + kH * kD * 4;
constexpr uint32_t kAuxCtl = kAuxPart + 10240;
// control words (32-bit): [0] arrival state, [1] first arrival, [8..16) shifted
// sink logits, [16..32) own (m, l)
constexpr uint32_t kLdsBytes = kAuxCtl + 128;
// One-launch step with a band: the first split to count in encodes the new
// token with four teams of four waves, in the table region (free once the
// split's partial is published): the teams' scratch, then their counters.
constexpr uint32_t kStepCtr = 4 * sizeof(step::Scratch<kD>);
static_assert(kStepCtr + 16 <= kLutBytes, "the step teams' scratch fits in the table region");

template <int WAVES>
constexpr uint32_t lds_bytes() {
  static_assert(WAVES * kMergeFloats * 4 <= kLutBytes, "merge scratch must fit in the table region");
  static_assert(WAVES >= 12, "8 table waves and 4 sink waves");
  static_assert(4 * kH * kD * 4 <= 10240 - kH * kD * 4, "combine outputs fit the part area");
  return kLdsBytes;
}

__device__ __forceinline__ size_t subtile_offset(const DecodeArgs &a, int b, int kv, int t_start, int bs_shift) {
  const int bs = a.layout.block_size;
  if (a.layout.block_table == nullptr && a.layout.blocks_per_seq == 1)
    return ((static_cast<size_t>(b) * a.num_kv_heads + kv) * bs + t_start) * kL;
  const int blk = bs_shift >= 0 ? (t_start >> bs_shift) : t_start / bs;
  const int row = t_start - blk * bs;
  const int logical = b * a.layout.blocks_per_seq + blk;
  const int phys = a.layout.block_table ? a.layout.block_table[logical] : logical;
  return ((static_cast<size_t>(phys) * a.num_kv_heads + kv) * bs + row) * kL;
}

// Thread t < 256 holds row (t mod 64) of t_v, columns 16 * (t / 64) .. +15.
template <bool TBF>
__device__ __forceinline__ void load_tv_rows(const DecodeArgs &a, const int kv, T4 (&tv)[4]) {
  const int tid = threadIdx.x;
  if (tid < 256) {
    const size_t row = (static_cast<size_t>(kv) * kD + (tid & (kD - 1))) * kD + 16 * (tid >> 6);
#pragma unroll
    for (int i = 0; i < 4; ++i) tv[i] = load_t4(a.t_v, row + 4 * i, TBF);
  }
}

// (BSTEP: the kernel's own instantiation, so that each kernel inlines a
// split pass of its own and the plain kernels compile as without the step)
template <int WAVES, bool KS, bool FP8, bool SQ, bool BSTEP, bool TBF>
__device__ __forceinline__ void split_pass(const DecodeArgs &a, uint8_t *smem, const int b, const int kv,
                                           const int t0, const int t1, const size_t row0, T4 (&tv)[4]) {
  const uint32_t sbase = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_u8_ptr)smem));
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = a.gqa;

  // ---- read-lane roles: rho = lane row, jj = group quad, tq = token of a pair, hh = head half
  const int rho = lane >> 4, jj = (lane >> 2) & 3, tq = (lane >> 1) & 1, hh = lane & 1;
  const int a2 = lane & 3;
  // ---- accumulator-lane roles: tau = lane row, column (set, head)
  const int set = (lane >> 3) & 1;

  uint32_t rselw = 0, kcw = 0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const uint32_t x = static_cast<uint32_t>((2 * (rho & 1) + tq) ^ t);  // byte of the group quad at step t
    rselw |= x << (8 * t);
    kcw |= static_cast<uint32_t>(16 * (4 * jj + x) + 8 * hh) << (8 * t);
  }
  const uint32_t vbase = sbase + kVBase + 8 * a2;

  float m_run = -INFINITY, l_run = 0.f;
  float z_run = 0.f;  // scalar value arm: sum of p * offset of the lane's tokens
  float4_t acc[4];
#pragma unroll
  for (int X = 0; X < 4; ++X) acc[X] = float4_t{0.f, 0.f, 0.f, 0.f};

  const int R0 = t0 & ~(kRound - 1);
  int nrounds = (t1 - R0 + kRound - 1) / kRound;
  const int last16 = (t1 - 1) & ~15;
  const uint8_t *kpool = a.k_codes;
  const uint8_t *vpool = a.v_codes;
  const int bsz = a.layout.block_size;
  const int bs_shift = (bsz & (bsz - 1)) == 0 ? __builtin_ctz(bsz) : -1;
  const uint32_t koff = (2 * rho + tq) * kL + 4 * jj;        // + 128 for odd r
  const uint32_t voff = (8 * (rho & 1) + 2 * jj) * kL + 4 * a2;  // + 16 for set 1

  // Code bytes of one round, per half h: K dwords kw[4h + r] (bytes 4jj..4jj+3
  // of tokens R + 32h + 8r + 2rho + tq) and V dwords vw[2h + s] (bytes
  // 4a2..4a2+3 of tokens R + 32h + 8rho + 2jj + s).
  // Key-scale format: lane l also loads the stored scale of token R + l,
  // issued after the code bytes; the scalar value arm loads that token's
  // (scale, offset) word the same way.
  auto load_round = [&](int R, uint32_t *kw, uint32_t *vw, uint32_t &ks, uint32_t &vq) {
    size_t sub[4];  // uniform: byte offsets of the round's four sub-tiles
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const size_t s0 = subtile_offset(a, b, kv, min(R + 32 * h, last16), bs_shift);
      const size_t s1 = subtile_offset(a, b, kv, min(R + 32 * h + 16, last16), bs_shift);
      sub[2 * h] = s0;
      sub[2 * h + 1] = s1;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint8_t *kb = kpool + (r < 2 ? s0 : s1);
        kw[4 * h + r] = *reinterpret_cast<const uint32_t *>(kb + koff + 128 * (r & 1));
      }
      const uint8_t *vb = vpool + ((rho >> 1) ? s1 : s0);
#pragma unroll
      for (int s = 0; s < 2; ++s) vw[2 * h + s] = *reinterpret_cast<const uint32_t *>(vb + voff + 16 * s);
    }
    if constexpr (KS || SQ) {
      const int st = lane >> 4;
      const size_t sl = st == 0 ? sub[0] : (st == 1 ? sub[1] : (st == 2 ? sub[2] : sub[3]));
      if constexpr (KS) ks = a.k_scales[sl / kL + (lane & 15)];
      if constexpr (SQ) vq = reinterpret_cast<const uint32_t *>(a.v_sq)[sl / kL + (lane & 15)];
    }
  };
  uint32_t kwb[kBuf][8], vwb[kBuf][4], ksb[kBuf] = {}, vqb[kBuf] = {};
#pragma unroll
  for (int k = 0; k < kBuf - 1; ++k)
    if (wave + k * WAVES < nrounds) load_round(R0 + kRound * (wave + k * WAVES), kwb[k], vwb[k], ksb[k], vqb[k]);

  // ---- setup: query transform, sink shifts, value codebook into LDS, table via MFMA
  {
    constexpr int NT = WAVES * 64;
    // thread (jq, e4) < 256 holds rows 4jq .. 4jq+3, columns 4e4 .. 4e4+3 of t_k_inv_t
    const int e4 = tid & 15, jq = tid >> 4;
    float qval = 0.f;
    T4 trow[4];
    if (tid < kH * kD) {
      const int qh = tid >> 6;
      if (qh < G) {
        const size_t qi = (row0 + qh) * kD + (tid & (kD - 1));
        qval = a.q_bf16 ? bf16_bits_to_float(static_cast<const uint16_t *>(a.q)[qi])
                        : static_cast<const float *>(a.q)[qi];
      }
    }
    if (tid < 256) {
      const size_t tk = (static_cast<size_t>(kv) * kD + 4 * jq) * kD + 4 * e4;
#pragma unroll
      for (int r = 0; r < 4; ++r) trow[r] = load_t4(a.t_k_inv_t, tk + r * kD, TBF);
    }
    constexpr int VPER = (kL * 256 + NT - 1) / NT;
    // codewords as raw words (fp16, or fp8 bytes converted where they are used)
    constexpr bool fp8 = FP8;
    const void *cbk = codebook_from(a.cb_k, fp8, static_cast<size_t>(kv) * kL * 256);
    const void *cbv = codebook_from(a.cb_v, fp8, static_cast<size_t>(kv) * kL * 256);
    // element e -> (g, c) so that each half-wave writes 32 distinct bank pairs
    auto vmap = [](int e, int &g, int &c) {
      const int r = e >> 5;
      g = 4 * ((e >> 3) & 3) + (r & 3);
      c = 8 * (r >> 2) + (e & 7);
    };
    uint2 vst[VPER];
    if constexpr (!SQ) {
#pragma unroll
      for (int k = 0; k < VPER; ++k) {
        const int e = tid + k * NT;
        if (e < kL * 256) {
          int g, c;
          vmap(e, g, c);
          vst[k] = codeword_raw(cbv, fp8, g * 256 + c);
        }
      }
    }
    // table waves: groups 8*(wave & 1) .. +7, codes 64*(wave >> 1) .. +63; 4-lane
    // block b = (group 8*(wave&1) + b/2, head half b&1)
    const bool lut_wave = wave < 8;
    const int blk = lane >> 2;
    const int lg = 8 * (wave & 1) + (blk >> 1);
    const int lh = blk & 1;
    const int lj = lane & 3;
    const int cbase = 64 * (wave >> 1);
    uint2 kst[16];
    if (lut_wave) {
#pragma unroll
      for (int t = 0; t < 16; ++t) kst[t] = codeword_raw(cbk, fp8, lg * 256 + cbase + 4 * t + lj);
    }
    // waves 8..11 form the shifted sink logits of heads 2(wave-8), 2(wave-8)+1
    const int sh = 2 * (wave - 8);
    float kbv = 0.f;
    if (wave >= 8) kbv = a.kbar[static_cast<size_t>(kv) * kD + lane];
    float *qs = reinterpret_cast<float *>(smem + kAuxQ);       // [8][64] query
    float *qsum = reinterpret_cast<float *>(smem + kAuxPart);  // [4 parts][8 heads][64] partial q'
    if (tid < kH * kD) qs[tid] = qval;
#pragma unroll
    for (int k = 0; k < VPER; ++k) {
      const int e = tid + k * NT;
      if (e < kL * 256) {
        int g, c;
        vmap(e, g, c);
        // scalar value arm: every group's table maps a code byte to its four
        // 2-bit codes (0..3, exact in fp16); the offsets are summed apart
        *reinterpret_cast<uint2 *>(smem + kVBase + (g & 3) * 8192 + (c << 5) + 8 * (g >> 2)) =
            SQ ? sq_unpack_f16(c) : codeword_f16(vst[k], fp8);
      }
    }
    __syncthreads();
    if (wave >= 8) {
      float *ctlf = reinterpret_cast<float *>(smem + kAuxCtl);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        if (sh + k < G) {
          const float dot = wave_sum(qs[(sh + k) * kD + lane] * kbv);
          if (lane == 0) ctlf[8 + sh + k] = a.sinks ? a.sinks[kv * G + sh + k] - a.scale * dot : -INFINITY;
        }
      }
    }
    if (tid < 256) {
      float4 acc4[kH];
#pragma unroll
      for (int hq = 0; hq < kH; ++hq) {
        const float4 q4 = *reinterpret_cast<const float4 *>(qs + hq * kD + 4 * jq);
        const float qq[4] = {q4.x, q4.y, q4.z, q4.w};
        acc4[hq] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float4 tr = t4_value(trow[r], TBF);
          acc4[hq].x = fmaf(qq[r], tr.x, acc4[hq].x);
          acc4[hq].y = fmaf(qq[r], tr.y, acc4[hq].y);
          acc4[hq].z = fmaf(qq[r], tr.z, acc4[hq].z);
          acc4[hq].w = fmaf(qq[r], tr.w, acc4[hq].w);
        }
      }
      // the 4 lane rows of a wave hold rows of the same columns: fold them, one part per wave
#pragma unroll
      for (int hq = 0; hq < kH; ++hq) {
        acc4[hq].x = add_rows32(add_rows16(acc4[hq].x));
        acc4[hq].y = add_rows32(add_rows16(acc4[hq].y));
        acc4[hq].z = add_rows32(add_rows16(acc4[hq].z));
        acc4[hq].w = add_rows32(add_rows16(acc4[hq].w));
        if (lane < 16) *reinterpret_cast<float4 *>(qsum + (wave * kH + hq) * kD + 4 * e4) = acc4[hq];
      }
    }
    __syncthreads();
    if (lut_wave) {
      float qv[4] = {0.f, 0.f, 0.f, 0.f};
      const int head = 4 * lh + lj;
      if (head < G) {
#pragma unroll
        for (int pp = 0; pp < 4; ++pp) {
          const float4 x4 = *reinterpret_cast<const float4 *>(qsum + (pp * kH + head) * kD + 4 * lg);
          qv[0] += x4.x; qv[1] += x4.y; qv[2] += x4.z; qv[3] += x4.w;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) qv[i] *= a.qscale;
      }
      half4_t a_hi, a_lo;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const _Float16 hi = static_cast<_Float16>(qv[i]);
        a_hi[i] = hi;
        a_lo[i] = static_cast<_Float16>(qv[i] - static_cast<float>(hi));
      }
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const half4_t bv = __builtin_bit_cast(half4_t, codeword_f16(kst[t], fp8));
        float4_t c = {0.f, 0.f, 0.f, 0.f};
        c = __builtin_amdgcn_mfma_f32_4x4x4f16(a_hi, bv, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_4x4x4f16(a_lo, bv, c, 0, 0, 0);
        half4_t o;
        o[0] = static_cast<_Float16>(c[0]);
        o[1] = static_cast<_Float16>(c[1]);
        o[2] = static_cast<_Float16>(c[2]);
        o[3] = static_cast<_Float16>(c[3]);
        // lane (group lg, half lh, code cbase + 4t + lj) holds heads 4lh .. 4lh+3
        *reinterpret_cast<half4_t *>(smem + (cbase + 4 * t + lj) * 256 + lg * 16 + 8 * lh) = o;
      }
    }
  }
  __syncthreads();

  // Selector of the key-side MFMA: row block r of the accumulator receives the
  // partials of tokens 8r + 2 rho + tq (A[m][k] = 1 where m = 4r + k-row).
  half8_t asel[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const _Float16 one = ((lane & 15) == 4 * r + rho) ? static_cast<_Float16>(1.f) : static_cast<_Float16>(0.f);
    asel[r] = half8_t{one, one, one, one, one, one, one, one};
  }

  auto process_round = [&](const int R, const uint32_t *kw, const uint32_t *vw, const uint32_t ks,
                           const uint32_t vq) {
    // K: both halves, four steps per token, pairs of steps per 16x16x32 MFMA
    uint32_t wr[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) wr[r] = __builtin_amdgcn_perm(kw[r], kw[r], rselw);
    float4_t kacc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int tp = 0; tp < 2; ++tp) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        half8_t e[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const uint32_t ta = 2 * tp, tb = 2 * tp + 1;
          const uint32_t w = wr[4 * h + r];
          const half4_t lo = tr16_read(sbase + __builtin_amdgcn_perm(w, kcw, 0x0C0C0000u | ((4u + ta) << 8) | ta));
          const half4_t hi = tr16_read(sbase + __builtin_amdgcn_perm(w, kcw, 0x0C0C0000u | ((4u + tb) << 8) | tb));
          e[r] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) kacc[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(asel[r], e[r], kacc[h], 0, 0, 0);
      }
    }
    // lane (tau, set, head): half h register i = token R + 32h + 8 tau + 2 i + set
    float z[8] = {kacc[0][0], kacc[0][1], kacc[0][2], kacc[0][3], kacc[1][0], kacc[1][1], kacc[1][2], kacc[1][3]};
    if constexpr (KS) {
      // the read path's per-token multiply: token R + l's scale is held by lane l
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int src = 32 * (i >> 2) + 8 * rho + 2 * (i & 3) + set;
        z[i] *= __uint_as_float(static_cast<uint32_t>(__shfl(static_cast<int>(ks), src)) << 16);
      }
    }
    // scalar value arm: (scale, offset) of the lane's tokens; the scale
    // carries 2^-8, so that the value product's B operand stays below 2^8 times it
    float vsc[8], vzr[8];
    if constexpr (SQ) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int src = 32 * (i >> 2) + 8 * rho + 2 * (i & 3) + set;
        const uint32_t w = static_cast<uint32_t>(__shfl(static_cast<int>(vq), src));
        vsc[i] = __uint_as_float(w << 16) * 0x1p-8f;
        vzr[i] = __uint_as_float(w & 0xffff0000u);
      }
    }
    if (R < t0 || R + kRound > t1) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int tok = R + 32 * (i >> 2) + 8 * rho + 2 * (i & 3) + set;
        if (tok < t0 || tok >= t1) {
          z[i] = -INFINITY;
          if constexpr (SQ) vsc[i] = vzr[i] = 0.f;  // rows past the tokens may hold anything
        }
      }
    }
    float zmax = fmaxf(fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3])), fmaxf(fmaxf(z[4], z[5]), fmaxf(z[6], z[7])));
    zmax = max_rows16(zmax);
    zmax = max_rows32(zmax);
    const float m_new = fmaxf(m_run, zmax);
    const bool bump = m_new > m_run + kLazyLog2;
    const float ref = bump ? m_new : m_run;
    const float alpha = bump ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.f;
    const float base = ref == -INFINITY ? 0.f : ref;
    float p[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) p[i] = __builtin_amdgcn_exp2f(z[i] - base);
    l_run = l_run * alpha + (((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7])));
    if constexpr (SQ)
      z_run = z_run * alpha + (((p[0] * vzr[0] + p[1] * vzr[1]) + (p[2] * vzr[2] + p[3] * vzr[3])) +
                               ((p[4] * vzr[4] + p[5] * vzr[5]) + (p[6] * vzr[6] + p[7] * vzr[7])));
    if (__any(bump && m_run != -INFINITY)) {
#pragma unroll
      for (int X = 0; X < 4; ++X) acc[X] *= alpha;
    }
    m_run = ref;
    const half4_t zero4 = {0, 0, 0, 0};
    // V: per half, tile X = coordinates of groups 4*(0..3) + X; sets 0 and 1 in one MFMA
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      half4_t pb;
#pragma unroll
      for (int i = 0; i < 4; ++i) pb[i] = static_cast<_Float16>(SQ ? p[4 * h + i] * vsc[4 * h + i] : p[4 * h + i]);
      const half8_t bpair = __builtin_shufflevector(set == 0 ? pb : zero4, set == 1 ? pb : zero4, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
      for (int X = 0; X < 4; ++X) {
        const uint32_t ca = (vw[2 * h] >> (8 * X)) & 0xffu;
        const uint32_t cb = (vw[2 * h + 1] >> (8 * X)) & 0xffu;
        const half4_t lo = tr16_read(vbase + (ca << 5) + X * 8192);
        const half4_t hi = tr16_read(vbase + (cb << 5) + X * 8192);
        const half8_t av = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        acc[X] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bpair, acc[X], 0, 0, 0);
      }
    }
  };

  for (int rd = wave; rd < nrounds; rd += kBuf * WAVES) {
#pragma unroll
    for (int k = 0; k < kBuf; ++k) {
      const int cur = rd + k * WAVES;
      if (cur >= nrounds) break;
      const int nxt = cur + (kBuf - 1) * WAVES;
      if (nxt < nrounds)
        load_round(R0 + kRound * nxt, kwb[(k + kBuf - 1) % kBuf], vwb[(k + kBuf - 1) % kBuf], ksb[(k + kBuf - 1) % kBuf],
                   vqb[(k + kBuf - 1) % kBuf]);
      process_round(R0 + kRound * cur, kwb[k], vwb[k], ksb[k], vqb[k]);
    }
  }
  load_tv_rows<TBF>(a, kv, tv);

  // ---- per-wave reduction: l over the rows of a column; the two set columns
  // of a head (lanes n and n + 8 of a row) are rescaled to a common max and summed
  float l_tot = add_rows32(add_rows16(l_run));
  const float m_head = fmaxf(m_run, row_ror<8>(m_run));
  const float wcol = (m_run == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run - m_head);
  l_tot *= wcol;
  l_tot += row_ror<8>(l_tot);
  float z_tot = 0.f;  // scalar value arm: the offsets' term of every coordinate of the head
  if constexpr (SQ) {
    z_tot = add_rows32(add_rows16(z_run)) * wcol;
    z_tot += row_ror<8>(z_tot);
  }
#pragma unroll
  for (int X = 0; X < 4; ++X) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float y = acc[X][i] * wcol;
      y += row_ror<8>(y);
      acc[X][i] = y;
    }
  }

  __syncthreads();  // every wave is done with the table before it becomes merge scratch
  float *merge = reinterpret_cast<float *>(smem + kMergeBase);
  float *mw = merge + wave * kMergeFloats;  // [0..8) m, [8..16) l, [16 + h*64 + d) acc
  const int head = lane & 7;
  if (lane < 8) {
    mw[head] = m_head;
    mw[kH + head] = l_tot;
  }
  if (set == 0) {
#pragma unroll
    for (int X = 0; X < 4; ++X)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        mw[2 * kH + head * kD + 4 * (4 * rho + X) + i] = SQ ? fmaf(acc[X][i], 256.f, z_tot) : acc[X][i];
  }
  __syncthreads();

  // ---- merge the waves into this split's partial (natural-log max), kept in LDS
  constexpr float kLn2 = 0.693147180559945309f;
  float *own = reinterpret_cast<float *>(smem + kAuxOwn);
  float *ownml = reinterpret_cast<float *>(smem + kAuxCtl) + 16;
  for (int i = tid; i < G * kD; i += WAVES * 64) {
    const int h = i / kD, d = i % kD;
    float big = -INFINITY;
    for (int w = 0; w < WAVES; ++w) big = fmaxf(big, merge[w * kMergeFloats + h]);
    float num = 0.f, den = 0.f;
    if (big != -INFINITY) {
      for (int w = 0; w < WAVES; ++w) {
        const float mwv = merge[w * kMergeFloats + h];
        const float wt = (mwv == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mwv - big);
        num = fmaf(wt, merge[w * kMergeFloats + 2 * kH + h * kD + d], num);
        den = fmaf(wt, merge[w * kMergeFloats + kH + h], den);
      }
    }
    own[i] = num;
    if (d == 0) {
      ownml[2 * h] = big == -INFINITY ? -INFINITY : big * kLn2;
      ownml[2 * h + 1] = den;
    }
  }
}

// Last split of a (sequence, KV head): log-sum-exp merge of the splits in
// index order, the sink once (shifted, Lemma S1), division, and out = s_hat t_v^T.
template <int WAVES, bool BSTEP, bool TBF>
__device__ __forceinline__ void combine_unit(const DecodeArgs &a, uint8_t *smem, const int b, const int kv,
                                             const size_t row0, const int own_split, const bool own_active,
                                             const int S, const int lo, const int tend, const int band_lo,
                                             const int sink_end, const T4 (&tv)[4]) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = a.gqa;
  // Sink-plus-recent band: positions [band_lo, sink_end) and [tend, S) (the
  // splits read [lo, tend) from the pools), attended here, in the table's
  // LDS region, and taken after the splits as one more partial.
  constexpr int kVW = 8;  // waves that sum the band's values
  using BL = BandLds<kD, kH, kVW>;
  const int nband = a.band_k ? max(0, sink_end - band_lo) + (S - tend) : 0;
  if constexpr (BSTEP) {
    // one-launch step: the new token is the band's last row, stored here and
    // read back after the barrier
    if (S > 0) {
      step::store_band_rows<kD>(a, b, kv, S - 1);
      __syncthreads();
    }
  }
  if (nband > 0) band_attention<kD, kH, WAVES, kVW>(a, smem, b, kv, row0, band_lo, sink_end, tend, S, 0, nband);
  float *bout = reinterpret_cast<float *>(smem + BL::kPart);  // [8][64] band term of the output
  float *shat = reinterpret_cast<float *>(smem + kAuxQ);    // [8][64]
  float *outp = reinterpret_cast<float *>(smem + kAuxOut);  // [4 parts][8 heads][64]
  float *ctlf = reinterpret_cast<float *>(smem + kAuxCtl);
  const float *own = reinterpret_cast<const float *>(smem + kAuxOwn);
  const int d = tid & (kD - 1), jp = tid >> 6;  // tv holds row d of t_v, columns 16*jp .. 16*jp+15
  if (!own_active) {  // the setup did not run: form the shifted sink logits here
    if (wave < G) {
      const size_t qi = (row0 + wave) * kD + lane;
      const float q0 = a.q_bf16 ? bf16_bits_to_float(static_cast<const uint16_t *>(a.q)[qi])
                                : static_cast<const float *>(a.q)[qi];
      const float dot = wave_sum(q0 * a.kbar[static_cast<size_t>(kv) * kD + lane]);
      if (lane == 0) ctlf[8 + wave] = a.sinks ? a.sinks[kv * G + wave] - a.scale * dot : -INFINITY;
    }
    __syncthreads();
  }
  if (tid < G * kD) {
    const int h = tid >> 6;
    const size_t r = (row0 + h) * a.n_split;
    const float sk = ctlf[8 + h];
    float big = sk, num = 0.f, den = sk == -INFINITY ? 0.f : 1.f;
    auto take = [&](float ms, float ls, float as) {
      if (ms == -INFINITY) return;
      if (ms > big) {
        const float f = big == -INFINITY ? 0.f : __expf(big - ms);
        num *= f;
        den *= f;
        big = ms;
      }
      const float w = __expf(ms - big);
      den = fmaf(w, ls, den);
      num = fmaf(w, as, num);
    };
    for (int s0 = 0; s0 < a.n_split; s0 += 8) {
      float ms[8], ls[8], as[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int sp = s0 + i;
        ms[i] = -INFINITY;
        ls[i] = 0.f;
        as[i] = 0.f;
        const bool nonempty = lo + sp * a.chunk < tend;
        if (sp == own_split) {
          if (own_active) {
            ms[i] = ctlf[16 + 2 * h];
            ls[i] = ctlf[16 + 2 * h + 1];
            as[i] = own[tid];
          }
        } else if (sp < a.n_split && nonempty) {
          ms[i] = load_dev(a.part_ml + 2 * (r + sp));
          ls[i] = load_dev(a.part_ml + 2 * (r + sp) + 1);
          as[i] = load_dev(a.part_acc + (r + sp) * kD + d);
        }
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) take(ms[i], ls[i], as[i]);
    }
    float bo = 0.f;
    if (nband > 0) {  // the band, after the splits
      const float *bst = reinterpret_cast<const float *>(smem + BL::kStat);
      const float mb = bst[h], lb = bst[kH + h];
      if (mb > big) {
        const float f = big == -INFINITY ? 0.f : __expf(big - mb);
        num *= f;
        den *= f;
        big = mb;
      }
      const float wb = __expf(mb - big);
      den = fmaf(wb, lb, den);
      bo = wb * reinterpret_cast<const float *>(smem + BL::kZ)[h * kD + d];
    }
    shat[tid] = den > 0.f ? num / den : 0.f;
    bout[tid] = den > 0.f ? bo / den : 0.f;
  } else if (tid < kH * kD) {
    shat[tid] = 0.f;
  }
  __syncthreads();
  if (tid < 256) {
    float o[kH];
#pragma unroll
    for (int h = 0; h < kH; ++h) o[h] = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int h = 0; h < kH; ++h) {
        const float4 sv = *reinterpret_cast<const float4 *>(shat + h * kD + 16 * jp + 4 * i);
        const float4 t = t4_value(tv[i], TBF);
        o[h] = fmaf(sv.x, t.x, o[h]);
        o[h] = fmaf(sv.y, t.y, o[h]);
        o[h] = fmaf(sv.z, t.z, o[h]);
        o[h] = fmaf(sv.w, t.w, o[h]);
      }
    }
#pragma unroll
    for (int h = 0; h < kH; ++h) outp[(jp * kH + h) * kD + d] = o[h];
  }
  __syncthreads();
  if (tid < G * kD) {
    const int h = tid >> 6;
    const float o = (outp[h * kD + d] + outp[(kH + h) * kD + d]) +
                    (outp[(2 * kH + h) * kD + d] + outp[(3 * kH + h) * kD + d]);
    a.out[(row0 + h) * kD + d] = nband > 0 ? o + bout[tid] : o;
  }
}

// One workgroup per (sequence, KV head, split); the arrival protocol is the
// one of the head_dim-128 kernel (relaxed agent-scope partials and counters,
// the last split combines, a split finding all others arrived does not publish).
// BSTEP: the one-launch step with a band (nova_kv_append_decode_attn): the new
// token is the band's last row, stored by the combining split; the first
// split to count in stores its codes (step_encode.h).
// TBF: the transforms are stored as bf16 (NOVA_KV_BF16_TRANSFORMS).
template <int WAVES, bool KS, bool FP8, bool SQ, bool BSTEP, bool TBF>
__global__ void __launch_bounds__(WAVES * 64) decode_lut_d64(DecodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[lds_bytes<WAVES>()];
  const int tid = threadIdx.x;
  // each XCD takes a contiguous range of the logical workgroup order
  int kv, b, split;
  unit_of_workgroup(xcd_contiguous(blockIdx.x, gridDim.x), a.n_split, a.b_chunk, a.num_kv_heads, kv, b, split);
  const int bk = b * a.num_kv_heads + kv;
  const int G = a.gqa;

  const int S = a.seq_lens[b];
  const int att_lo = a.window > 0 ? max(0, S - a.window) : 0;
  // the pools are read for [lo, tend): the attended span without the band
  const AttendedSpans spn = attended_spans(att_lo, S, a.n_sink, a.n_rec);
  const int lo = spn.code_lo, tend = spn.code_hi;
  const int t0 = lo + split * a.chunk;  // splits tile the span read from the pools
  const int t1 = min(tend, lo + (split + 1) * a.chunk);
  const size_t row0 = static_cast<size_t>(b) * a.num_q_heads + kv * G;
  const bool active = t0 < t1;

  T4 tv[4];
  if (active) {
    split_pass<WAVES, KS, FP8, SQ, BSTEP, TBF>(a, smem, b, kv, t0, t1, row0, tv);
  } else {
    load_tv_rows<TBF>(a, kv, tv);
  }
  // Arrival: every split publishes its partial (when it has one) and counts
  // itself in; the split that brings the count to n_split combines.  The
  // protocol runs in waves 4.. (thread kCtl and the publishing threads), which
  // hold no loads of t_v: a wave's memory operations complete in issue order,
  // so a wait there would also wait for t_v.
  constexpr int kCtl = 256;
  int *ctl = reinterpret_cast<int *>(smem + kAuxCtl);
  __syncthreads();
  if (a.n_split > 1) {
    if (tid >= kCtl) {
      if (active) {
        const float *own = reinterpret_cast<const float *>(smem + kAuxOwn);
        const float *ownml = reinterpret_cast<const float *>(smem + kAuxCtl) + 16;
        for (int i = tid - kCtl; i < G * kD; i += WAVES * 64 - kCtl) {
          const int h = i / kD, d = i % kD;
          const size_t r = (row0 + h) * a.n_split + split;
          store_dev(a.part_acc + r * kD + d, own[i]);
          if (d == 0) {
            store_dev(a.part_ml + 2 * r, ownml[2 * h]);
            store_dev(a.part_ml + 2 * r + 1, ownml[2 * h + 1]);
          }
        }
      }
      __builtin_amdgcn_s_waitcnt(0);  // this thread's partial stores have completed
    }
    __syncthreads();
    if (tid == kCtl) {
      if constexpr (BSTEP) {
        const int old = __hip_atomic_fetch_add(a.counters + bk, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (old == a.n_split - 1) __hip_atomic_store(a.counters + bk, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ctl[0] = old == a.n_split - 1;
        ctl[1] = old == 0;
      } else {
        const int last = __hip_atomic_fetch_add(a.counters + bk, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                         a.n_split - 1;
        if (last) __hip_atomic_store(a.counters + bk, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ctl[0] = last;
      }
    }
    __syncthreads();
    if constexpr (!BSTEP) {
      if (ctl[0] == 0) return;
    }
  }
  if constexpr (BSTEP) {
    // the first split to count in (the only one without splits) encodes the
    // new token while the others finish: team tid / 256 takes tasks team,
    // team + 4, ...
    if ((a.n_split == 1 || ctl[1] != 0) && S > 0) {
      int *ctr = reinterpret_cast<int *>(smem + kStepCtr);
      if (tid < 4) ctr[tid] = 0;
      __syncthreads();
      const int team = tid >> 8, p = S - 1;
      const int bsz = a.layout.block_size;
      const int bs_shift = (bsz & (bsz - 1)) == 0 ? __builtin_ctz(bsz) : -1;
      const size_t tokoff = subtile_offset(a, b, kv, p & ~15, bs_shift) + static_cast<size_t>(p & 15) * kL;
      int phase = 0;  // shared by every copy of the meeting
      auto meet = [&] { step::team_meet(ctr + team, ++phase); };
      step::encode_token<kD, KS, SQ, TBF>(a, reinterpret_cast<step::Scratch<kD> *>(smem)[team], b, kv, team, 4, tokoff,
                                     tid & 255, FP8, meet);
      __syncthreads();  // the table region is free again
    }
    if (a.n_split > 1 && ctl[0] == 0) return;
  }
  combine_unit<WAVES, BSTEP, TBF>(a, smem, b, kv, row0, split, active, S, lo, tend, att_lo, spn.sink_end, tv);
}

}  // namespace

template <bool BSTEP, bool TBF>
void launch_d64(const DecodeArgs &a, const dim3 grid, const dim3 block, hipStream_t stream) {
  constexpr int W = 16;
  if (a.v_sq) {  // the scalar value arm (keys in either codebook format)
    if (a.k_scales)
      a.cb_fp8 ? decode_lut_d64<W, true, true, true, BSTEP, TBF><<<grid, block, 0, stream>>>(a)
               : decode_lut_d64<W, true, false, true, BSTEP, TBF><<<grid, block, 0, stream>>>(a);
    else
      a.cb_fp8 ? decode_lut_d64<W, false, true, true, BSTEP, TBF><<<grid, block, 0, stream>>>(a)
               : decode_lut_d64<W, false, false, true, BSTEP, TBF><<<grid, block, 0, stream>>>(a);
  } else if (a.k_scales) {
    a.cb_fp8 ? decode_lut_d64<W, true, true, false, BSTEP, TBF><<<grid, block, 0, stream>>>(a)
             : decode_lut_d64<W, true, false, false, BSTEP, TBF><<<grid, block, 0, stream>>>(a);
  } else {
    a.cb_fp8 ? decode_lut_d64<W, false, true, false, BSTEP, TBF><<<grid, block, 0, stream>>>(a)
             : decode_lut_d64<W, false, false, false, BSTEP, TBF><<<grid, block, 0, stream>>>(a);
  }
}

hipError_t launch_decode_lut64(const DecodeArgs &a, hipStream_t stream) {
  // 16 waves, 4 per SIMD: the kernel fits in 128 VGPRs.  A step (append) runs
  // here only with a band whose recent part holds the new token.
  if (a.append && !(a.band_k && a.n_rec >= 1)) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(a.batch * a.num_kv_heads * a.n_split));
  const dim3 block(16 * 64);
  if (a.t_bf16)
    a.append ? launch_d64<true, true>(a, grid, block, stream) : launch_d64<false, true>(a, grid, block, stream);
  else
    a.append ? launch_d64<true, false>(a, grid, block, stream) : launch_d64<false, false>(a, grid, block, stream);
  return hipGetLastError();
}

}  // namespace novakv
