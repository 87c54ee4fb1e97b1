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
//   tm  = side transform of the KV head ([D][D], row-major; fp32, or bf16
//         bit patterns when tbf, kept as loaded and converted where used)
//   cb, fp8, cw0 = side codebooks ([Hkv][L][256] codewords, fp16 or fp8) and
//         the index of the KV head's first codeword; the raw words are kept
//         and converted where they are used
template <int D>
__device__ __forceinline__ void load_rows(const int t, const void *tm, const int tbf, const int blk,
                                          T4 (&trow)[D / 32]) {
  constexpr int RPT = D / 32;
  const int rg = t >> 3, c4 = t & 7;
  const size_t col = kCols * blk + 4 * c4;
#pragma unroll
  for (int j = 0; j < RPT; ++j) trow[j] = load_t4(tm, col + static_cast<size_t>(RPT * rg + j) * D, tbf);
}
__device__ __forceinline__ void load_codewords(const int t, const void *cb, const bool fp8, const size_t cw0,
                                               const int blk, uint2 (&cw)[kPer]) {
  const int gl = t >> 5, r = t & 31;
  const size_t row = cw0 + static_cast<size_t>(kGroups * blk + gl) * kCodebookSize;
#pragma unroll
  for (int k = 0; k < kPer; ++k) cw[k] = codeword_raw(cb, fp8, row + r + 32 * k);
}
template <int D>
__device__ __forceinline__ void load_block(const int t, const void *tm, const int tbf, const void *cb,
                                           const bool fp8, const size_t cw0, const int blk, T4 (&trow)[D / 32],
                                           uint2 (&cw)[kPer]) {
  load_rows<D>(t, tm, tbf, blk, trow);
  load_codewords(t, cb, fp8, cw0, blk, cw);
}

// Phase 2 (after x is in LDS): this wave's share of the 32 coefficients.
template <int D>
__device__ __forceinline__ void partial_block(const int t, Scratch<D> &s, const T4 (&trow)[D / 32], const int tbf) {
  constexpr int RPT = D / 32;
  const int rg = t >> 3, c4 = t & 7;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const double x = s.xs[RPT * rg + j];
    const float4 tr = t4_value(trow[j], tbf);
    acc[0] = fma(x, static_cast<double>(tr.x), acc[0]);
    acc[1] = fma(x, static_cast<double>(tr.y), acc[1]);
    acc[2] = fma(x, static_cast<double>(tr.z), acc[2]);
    acc[3] = fma(x, static_cast<double>(tr.w), acc[3]);
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

// bf16 bit pattern of an fp64 value: rounded to fp32, then to bf16, each to
// nearest even.
__device__ __forceinline__ uint16_t bf16_of(const double x) {
  const uint32_t f = __float_as_uint(static_cast<float>(x));
  return static_cast<uint16_t>((f + 0x7fffu + ((f >> 16) & 1u)) >> 16);
}

// All D coefficients of one token (x in s.xs) into u[D]: block after block,
// each with the block's own arithmetic (partial_block, then coefficient), the
// next block's transform rows requested while the current one is summed.
// `first` holds block 0's rows (load_rows) on entry.  Two meetings of the
// team (sync) per block.
template <int D, class Sync>
__device__ __forceinline__ void token_coefficients(const int t, Scratch<D> &s, const void *tm, const int tbf,
                                                   T4 (&first)[D / 32], double *u, Sync sync) {
  constexpr int NB = D / kCols;
  T4 next[D / 32];
#pragma unroll
  for (int bb = 0; bb < NB; ++bb) {
    if (bb + 1 < NB) load_rows<D>(t, tm, tbf, bb + 1, next);
    partial_block<D>(t, s, first, tbf);
    sync();
    if (t < kCols) u[kCols * bb + t] = coefficient<D>(s, t);
    sync();
    if (bb + 1 < NB) {
#pragma unroll
      for (int j = 0; j < D / 32; ++j) first[j] = next[j];
    }
  }
}

// Scalar value arm of one token (paper: Sec. "Bit rate" and the
// implementation table: per-token affine INT2 values with a BF16 scale and
// offset) from its D coefficients u: offset = bf16(min), scale =
// bf16((max - min) / 3), and level_i = clamp(round_half_even((u_i - offset)
// / scale), 0, 3) with the stored values (0 when the stored scale is 0),
// into q[i].  Thread t < D takes coordinate t; D is a multiple of 64, so
// the waves that hold coordinates are whole.  red: 2 D / 64 doubles of LDS.
// Two meetings of the team (sync).
template <int D, class Sync>
__device__ __forceinline__ void sq_levels(const int t, const double *u, double *red, uint8_t *q, Sync sync,
                                          uint16_t &scale_bits, uint16_t &offset_bits) {
  static_assert(D % 64 == 0, "whole waves hold the coordinates");
  double mn = t < D ? u[t] : 0.0, mx = mn;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    mn = fmin(mn, __shfl_xor(mn, o, 64));
    mx = fmax(mx, __shfl_xor(mx, o, 64));
  }
  if (t < D && (t & 63) == 0) {
    red[t >> 6] = mn;
    red[D / 64 + (t >> 6)] = mx;
  }
  sync();
  mn = red[0];
  mx = red[D / 64];
#pragma unroll
  for (int w = 1; w < D / 64; ++w) {
    mn = fmin(mn, red[w]);
    mx = fmax(mx, red[D / 64 + w]);
  }
  offset_bits = bf16_of(mn);
  scale_bits = bf16_of((mx - mn) / 3.0);
  const double zero = bf16_bits_to_float(offset_bits), scale = bf16_bits_to_float(scale_bits);
  if (t < D) q[t] = scale > 0.0 ? static_cast<uint8_t>(fmin(fmax(rint((u[t] - zero) / scale), 0.0), 3.0)) : 0;
  sync();
}

// Byte g of a token's scalar-arm codes: levels 4g + j at bits 2j, 2j + 1.
__device__ __forceinline__ uint8_t sq_byte(const uint8_t *q, const int g) {
  return static_cast<uint8_t>(q[4 * g] | (q[4 * g + 1] << 2) | (q[4 * g + 2] << 4) | (q[4 * g + 3] << 6));
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


}  // namespace encblk
}  // namespace novakv
