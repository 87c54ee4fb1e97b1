// The new token's encode inside the one-launch decode step when the call
// has a sink-plus-recent band whose recent part holds that token.
//
// Paper: Algorithm 1 (the write of the new token, then the attention), Sec.
// "Sink-plus-recent band" (the newest positions are held in BF16 and
// attended exactly), Sec. "Bit rate" (keys as VQ codes with a per-token BF16
// scale, values as per-token affine INT2).
//
// The new token is the band's last row, so the attention needs none of its
// codes: the encode only stores them (codes, and in the key-scale format the
// scale, in the scalar value arm the levels and (scale, offset)), exactly as
// the one-token encoder does.  Its work is a list of tasks, run by teams of
// 256 threads (4 whole waves) that meet through an LDS arrival counter:
//   keys:   one block item per 8 groups, or with the key scale one task (all
//           D coefficients, rho, then every block's codes of u / rho);
//   values: one block item per 8 groups, or in the scalar arm one task (all
//           D coefficients, min and max, levels).
// Every task does the one-token encoder's arithmetic (encode_block.h), so
// both paths store the same bytes.
#pragma once

#include "encode_block.h"
#include "nova_kv_internal.h"

namespace novakv {
namespace step {

// All four waves of a team arrive, then each continues once the counter has
// reached 4 * phase: LDS writes before the call are visible after it.
__device__ __forceinline__ void team_meet(int *ctr, const int phase) {
  if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
  while (__hip_atomic_load(ctr, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < 4 * phase)
    __builtin_amdgcn_s_sleep(1);
}

template <int D, bool KS, bool SQ>
struct Tasks {
  static constexpr int kBlocks = D / kGroupDim / encblk::kGroups;
  static constexpr int kKey = KS ? 1 : kBlocks;
  static constexpr int kAll = kKey + (SQ ? 1 : kBlocks);
  // meetings of task j: its x, then two per block of coefficients and one for
  // rho (key scale) or two for the levels (scalar arm); a block item meets twice
  __device__ static int phases(const int j) {
    if (j < kKey) return KS ? 2 + 2 * kBlocks : 2;
    return SQ ? 3 + 2 * kBlocks : 2;
  }
  // a team's meetings for tasks first, first + stride, ..., with the last one
  // after its last task
  __device__ static int phases_of(const int first, const int stride) {
    int n = 1;
    for (int j = first; j < kAll; j += stride) n += phases(j);
    return n;
  }
};

// LDS of one team: two sets of scratch that successive tasks alternate
// between, so no meeting guards their reuse.
template <int D>
struct Scratch {
  encblk::Scratch<D> sc[2];
  double u[2][D];              // a whole-token task's coefficients
  double red[2][2 * D / 64];   // its min and max words
  uint8_t q[2][D];             // its scalar-arm levels
};

// Tasks first, first + stride, ... of the new token at code row offset tokoff
// of the pools, by team thread t (0..255); meet() is the team's meeting.
// TBF: the transforms are stored as bf16.
template <int D, bool KS, bool SQ, bool TBF, class Meet>
__device__ __forceinline__ void encode_token(const DecodeArgs &a, Scratch<D> &ls, const int b, const int kv,
                                             const int first, const int stride, const size_t tokoff, const int t,
                                             const bool fp8, Meet meet) {
  using T = Tasks<D, KS, SQ>;
  constexpr int L = D / kGroupDim;
  const size_t elem = (static_cast<size_t>(b) * a.num_kv_heads + kv) * D + (t & (D - 1));
  auto element = [&](const bool key) {  // element t of the token minus k_bar (keys) or of the token (values)
    const void *src = key ? a.k_new : a.v_new;
    double x = a.new_bf16 ? static_cast<double>(bf16_bits_to_float(static_cast<const uint16_t *>(src)[elem]))
                          : static_cast<double>(static_cast<const float *>(src)[elem]);
    if (key) x -= static_cast<double>(a.kbar[kv * D + t]);
    return x;
  };
  const size_t cw0 = static_cast<size_t>(kv) * L * kCodebookSize;
  int k = 0;
  for (int j = first; j < T::kAll; j += stride, ++k) {
    encblk::Scratch<D> &s = ls.sc[k & 1];
    double *u = ls.u[k & 1];
    const bool key = j < T::kKey;
    const void *tm = transform_of(key ? a.t_k : a.t_v, kv, D, TBF);
    const void *cb = key ? a.cb_k : a.cb_v;
    T4 rows[D / 32];
    uint2 cw[encblk::kPer];
    if ((key && KS) || (!key && SQ)) {
      encblk::load_rows<D>(t, tm, TBF, 0, rows);
      if (key) encblk::load_codewords(t, cb, fp8, cw0, 0, cw);
      if (t < D) s.xs[t] = element(key);
      meet();
      encblk::token_coefficients<D>(t, s, tm, TBF, rows, u, meet);
      if (key) {
        // rho, then the blocks' codes of the coefficients divided by it (the
        // next block's codewords requested while one block is searched)
        if (t == 0) s.wpart[0][0] = encblk::key_scale<D>(u);
        meet();
        const double rho = s.wpart[0][0];
#pragma unroll
        for (int bb = 0; bb < T::kBlocks; ++bb) {
          uint2 nx[encblk::kPer];
          if (bb + 1 < T::kBlocks) encblk::load_codewords(t, cb, fp8, cw0, bb + 1, nx);
          double uu[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const double v = u[encblk::kCols * bb + 4 * (t >> 5) + i];
            uu[i] = rho > 0.0 ? v / rho : 0.0;
          }
          const int code = encblk::search_codes(t, uu, cw, fp8);
          if ((t & 31) == 0) a.k_codes_w[tokoff + encblk::kGroups * bb + (t >> 5)] = static_cast<uint8_t>(code);
          if (bb + 1 < T::kBlocks) {
#pragma unroll
            for (int i = 0; i < encblk::kPer; ++i) cw[i] = nx[i];
          }
        }
        if (t == 0) a.k_scales_w[tokoff / L] = encblk::bf16_of(rho);
      } else {
        uint16_t sbits, zbits;
        encblk::sq_levels<D>(t, u, ls.red[k & 1], ls.q[k & 1], meet, sbits, zbits);
        if (t < L) a.v_codes_w[tokoff + t] = encblk::sq_byte(ls.q[k & 1], t);
        if (t == 0) {
          a.v_sq_w[(tokoff / L) * 2] = sbits;
          a.v_sq_w[(tokoff / L) * 2 + 1] = zbits;
        }
      }
    } else {
      const int blk = key ? j : j - T::kKey;
      encblk::load_block<D>(t, tm, TBF, cb, fp8, cw0, blk, rows, cw);
      if (t < D) s.xs[t] = element(key);
      meet();
      encblk::partial_block<D>(t, s, rows, TBF);
      meet();
      const int code = encblk::search_block<D>(t, s, cw, fp8);
      if ((t & 31) == 0)
        (key ? a.k_codes_w : a.v_codes_w)[tokoff + encblk::kGroups * blk + (t >> 5)] = static_cast<uint8_t>(code);
    }
  }
  meet();  // every read of the scratch is done
}

// The new token's key and value rows (bf16: as given, or an fp32 element
// rounded to nearest even) into its band slot, by threads 0 .. 2D-1.
template <int D>
__device__ __forceinline__ void store_band_rows(const DecodeArgs &a, const int b, const int kv, const int pos) {
  const int tid = threadIdx.x;
  if (tid >= 2 * D) return;
  const int side = tid / D, d = tid % D;
  const void *src = side ? a.v_new : a.k_new;
  const size_t idx = (static_cast<size_t>(b) * a.num_kv_heads + kv) * D + d;
  uint16_t bits;
  if (a.new_bf16) {
    bits = static_cast<const uint16_t *>(src)[idx];
  } else {
    const uint32_t f = __float_as_uint(static_cast<const float *>(src)[idx]);
    bits = static_cast<uint16_t>((f + 0x7fffu + ((f >> 16) & 1u)) >> 16);
  }
  const int nb = a.n_sink + a.n_rec;
  (side ? a.band_v_w : a.band_k_w)[((static_cast<size_t>(b) * a.num_kv_heads + kv) * nb +
                                    band_slot(pos, a.n_sink, a.n_rec)) * D + d] = bits;
}

}  // namespace step
}  // namespace novakv
