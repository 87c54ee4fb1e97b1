// One block of the append-time encoder: 8 groups (32 transform coordinates)
// of one token on one side (keys or values), computed by a team of 256
// threads made of 4 whole waves.  Shared by the one-token encoder and the
// fused append-and-decode step, so both store identical codes.
//
// Paper: Algorithm 1 (write step, Q+((k - k_bar) R_K)), Theorem 1 (key
// transform), Corollary 1 (s = v R_V), Sec. "Calibration" (each group gets
// the codeword at the smallest squared distance in the transform domain).
// The transform and the distances are evaluated in fp64; the stored index is
// the argmin, smallest index among equal distances.
//
// Team thread t: transform role (rg, c4) = (t >> 3, t & 7) owns rows
// (D/32) rg .. (D/32) rg + D/32 - 1 of columns 4 c4 .. 4 c4 + 3; search role
// (gl, r) = (t >> 5, t & 31) scans codewords r + 32 k of group gl.
// Column sums are fixed in order: an fp64 fma chain over a thread's rows,
// then a butterfly over the 8 row groups of a wave (lanes 8, 16, 32 apart,
// the value of lane c4 kept), then the 4 waves' partials added in order by
// each searching thread.
#pragma once

#include "nova_kv_internal.h"

namespace novakv {
namespace encblk {

constexpr int kTeam = 256;
constexpr int kGroups = 8;                        // groups per block
constexpr int kCols = kGroups * kGroupDim;        // 32 coordinates
constexpr int kPer = kCodebookSize / 32;          // codewords per search lane

// LDS of one team: x [D] doubles, wave partials [4][32] doubles.
template <int D>
struct Scratch {
  double xs[D];
  double wpart[4][kCols];
};

// Phase 1 (issue only): the block's transform columns and codewords.
//   tm  = side transform of the KV head ([D][D] fp32, row-major)
//   cb, fp8, cw0 = side codebooks ([Hkv][L][256] codewords, fp16 or fp8) and
//         the index of the KV head's first codeword; the raw words are kept
//         and converted where they are used
template <int D>
__device__ __forceinline__ void load_rows(const int t, const float *tm, const int blk, float4 (&trow)[D / 32]) {
  constexpr int RPT = D / 32;
  const int rg = t >> 3, c4 = t & 7;
  const float *col = tm + kCols * blk + 4 * c4;
#pragma unroll
  for (int j = 0; j < RPT; ++j) trow[j] = *reinterpret_cast<const float4 *>(col + (RPT * rg + j) * D);
}
__device__ __forceinline__ void load_codewords(const int t, const void *cb, const bool fp8, const size_t cw0,
                                               const int blk, uint2 (&cw)[kPer]) {
  const int gl = t >> 5, r = t & 31;
  const size_t row = cw0 + static_cast<size_t>(kGroups * blk + gl) * kCodebookSize;
#pragma unroll
  for (int k = 0; k < kPer; ++k) cw[k] = codeword_raw(cb, fp8, row + r + 32 * k);
}
template <int D>
__device__ __forceinline__ void load_block(const int t, const float *tm, const void *cb, const bool fp8,
                                           const size_t cw0, const int blk, float4 (&trow)[D / 32],
                                           uint2 (&cw)[kPer]) {
  load_rows<D>(t, tm, blk, trow);
  load_codewords(t, cb, fp8, cw0, blk, cw);
}

// Phase 2 (after x is in LDS): this wave's share of the 32 coefficients.
template <int D>
__device__ __forceinline__ void partial_block(const int t, Scratch<D> &s, const float4 (&trow)[D / 32]) {
  constexpr int RPT = D / 32;
  const int rg = t >> 3, c4 = t & 7;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const double x = s.xs[RPT * rg + j];
    acc[0] = fma(x, static_cast<double>(trow[j].x), acc[0]);
    acc[1] = fma(x, static_cast<double>(trow[j].y), acc[1]);
    acc[2] = fma(x, static_cast<double>(trow[j].z), acc[2]);
    acc[3] = fma(x, static_cast<double>(trow[j].w), acc[3]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    double v = acc[i];
    v = v + __shfl_xor(v, 8, 64);
    v = v + __shfl_xor(v, 16, 64);
    v = v + __shfl_xor(v, 32, 64);
    acc[i] = v;
  }
  if ((t & 63) < 8) {
#pragma unroll
    for (int i = 0; i < 4; ++i) s.wpart[t >> 6][4 * c4 + i] = acc[i];
  }
}

// Nearest codeword of group t >> 5 to the coefficients u, returned in all 32
// lanes of the group: fp64 distances, the smallest index among equal ones.
__device__ __forceinline__ int search_codes(const int t, const double (&u)[4], const uint2 (&cw)[kPer],
                                            const bool fp8) {
  const int r = t & 31;
  const double u0 = u[0], u1 = u[1], u2 = u[2], u3 = u[3];
  double best = INFINITY;
  int arg = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
#pragma clang fp contract(off)
    const int c = r + 32 * k;
    const uint2 w = codeword_f16(cw[k], fp8);
    const double e0 = u0 - static_cast<double>(half_bits_to_float(static_cast<uint16_t>(w.x & 0xffff)));
    const double e1 = u1 - static_cast<double>(half_bits_to_float(static_cast<uint16_t>(w.x >> 16)));
    const double e2 = u2 - static_cast<double>(half_bits_to_float(static_cast<uint16_t>(w.y & 0xffff)));
    const double e3 = u3 - static_cast<double>(half_bits_to_float(static_cast<uint16_t>(w.y >> 16)));
    double dist = e0 * e0;
    dist = dist + e1 * e1;
    dist = dist + e2 * e2;
    dist = dist + e3 * e3;
    if (dist < best) {
      best = dist;
      arg = c;
    }
  }
#pragma unroll
  for (int o = 16; o > 0; o >>= 1) {
    const double ob = __shfl_xor(best, o, 64);
    const int oa = __shfl_xor(arg, o, 64);
    if (ob < best || (ob == best && oa < arg)) {
      best = ob;
      arg = oa;
    }
  }
  return arg;
}

// Column c of the block: the 4 waves' partials added in wave order.
template <int D>
__device__ __forceinline__ double coefficient(const Scratch<D> &s, const int c) {
  return ((s.wpart[0][c] + s.wpart[1][c]) + s.wpart[2][c]) + s.wpart[3][c];
}

// Phase 3 (after the partials are in LDS): nearest codeword of group t >> 5,
// returned in all 32 lanes of the group.
template <int D>
__device__ __forceinline__ int search_block(const int t, const Scratch<D> &s, const uint2 (&cw)[kPer],
                                            const bool fp8) {
  const int gl = t >> 5;
  double uu[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) uu[i] = coefficient<D>(s, gl * 4 + i);
  return search_codes(t, uu, cw, fp8);
}

// Key-scale format: rho = sqrt(sum of the squared coefficients, added in
// coordinate order) / sqrt(D), each square rounded before it is added.
template <int D>
__device__ __forceinline__ double key_scale(const double *u) {
  double s = 0.0;
  for (int i = 0; i < D; ++i) {
#pragma clang fp contract(off)
    s = s + u[i] * u[i];
  }
  return sqrt(s) / sqrt(static_cast<double>(D));
}

// bf16 bit pattern of rho: rounded to fp32, then to bf16, each to nearest even.
__device__ __forceinline__ uint16_t bf16_of(const double x) {
  const uint32_t f = __float_as_uint(static_cast<float>(x));
  return static_cast<uint16_t>((f + 0x7fffu + ((f >> 16) & 1u)) >> 16);
}

}  // namespace encblk
}  // namespace novakv
