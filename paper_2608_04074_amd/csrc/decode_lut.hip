// Decode stage 1 for head_dim 128 and up to 4 query heads per KV head.
//
// One workgroup owns one (sequence, KV head, context split) unit.  It stages
// the KV head's value codebook in LDS and builds a per-query table of partial
// logits LUT[c][g] = (q'_h[4g..4g+3] . C_K[g][c])_{h<4} (fp16, 64 KB) with
// MFMA, so that a key's logit is the sum of its 32 table entries.  This is
// the paper's read path (q' = q R_K^{-T} folded in once per step, one
// codebook lookup per group; Sec. "Decoding kernel and read path") with the
// q'-codeword dot products hoisted out of the token loop.
//
// Token loop, per wave, per round of 64 tokens:
//  * K: ds_read_b64_tr_b16 gathers from the table.  Lane (beta,u,v) =
//    16*beta + 4*u + v reads, at step t, group 8u + ((t + 2v + (beta&1)) & 7)
//    of token 16r + 4*beta + v: the 32 lanes of each half-wave touch 32
//    distinct groups, i.e. 32 distinct bank pairs of the entry-major table.
//    The transposing read hands lane (beta,u,v) the four partials of
//    (token 16r + 4*beta + u, head v), summed with v_dot2_f32_f16.
//  * online softmax in log2 units (q' carries the log2(e) factor);
//  * V: transposing reads of the staged codebook give the token-major MFMA
//    operand (4 tokens of one transform coordinate per lane); the
//    probabilities already sit in the matching layout.  One
//    v_mfma_f32_16x16x16_f16 per (token set, 16 coordinates).
// The value accumulator stays in the transform domain (Corollary 1); the
// combine kernel applies t_v^T once per head.
#include <math.h>

#include "nova_kv_internal.h"

namespace novakv {

namespace {

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4_t *lds_short4_ptr;
typedef __attribute__((address_space(3))) uint8_t *lds_u8_ptr;

constexpr int kD = 128;
constexpr int kL = kD / kGroupDim;          // 32 groups
constexpr uint32_t kLutBytes = 65536;       // [256 codes][32 groups][4 heads] fp16
constexpr uint32_t kVBase = kLutBytes;      // value codebook, 64 KB
constexpr uint32_t kMergeBase = 0;          // per-wave merge scratch, reuses the table once done
constexpr int kMergeFloats = 4 * kD + 8;

template <int WAVES>
constexpr uint32_t lds_bytes() {
  static_assert(WAVES * kMergeFloats * 4 <= kLutBytes, "merge scratch must fit in the table region");
  static_assert(WAVES >= kL / 4, "one wave per group block builds the table");
  return 2 * 65536;
}

__device__ __forceinline__ half4_t tr16_read(uint32_t addr) {
  const short4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4_ptr)(uintptr_t)(addr));
  return __builtin_bit_cast(half4_t, v);
}

__device__ __forceinline__ float sum4(half4_t v, float acc) {
  const half2_t ones = {(_Float16)1.0f, (_Float16)1.0f};
  const half2_t lo = {v[0], v[1]};
  const half2_t hi = {v[2], v[3]};
  acc = __builtin_amdgcn_fdot2(lo, ones, acc, false);
  return __builtin_amdgcn_fdot2(hi, ones, acc, false);
}

// Cross-row reductions (lane ^ 16, lane ^ 32) with v_permlane{16,32}_swap:
// swapping x with a copy of itself yields (rows 0,2 | rows 1,3), or (low half |
// high half), in the two results, whose elementwise combination is the
// reduction.  The two results are copied out of the returned vector before any
// bit cast (a bit cast of a vector element reads element 0 with this compiler).
struct SwapPair {
  float a, b;
};
__device__ __forceinline__ SwapPair swap_rows16(float x) {
  const unsigned xu = __builtin_bit_cast(unsigned, x);
  const auto s = __builtin_amdgcn_permlane16_swap(xu, xu, false, false);
  const unsigned s0 = s[0], s1 = s[1];
  return {__builtin_bit_cast(float, s0), __builtin_bit_cast(float, s1)};
}
__device__ __forceinline__ SwapPair swap_rows32(float x) {
  const unsigned xu = __builtin_bit_cast(unsigned, x);
  const auto s = __builtin_amdgcn_permlane32_swap(xu, xu, false, false);
  const unsigned s0 = s[0], s1 = s[1];
  return {__builtin_bit_cast(float, s0), __builtin_bit_cast(float, s1)};
}
__device__ __forceinline__ float max_rows16(float x) { const SwapPair p = swap_rows16(x); return fmaxf(p.a, p.b); }
__device__ __forceinline__ float max_rows32(float x) { const SwapPair p = swap_rows32(x); return fmaxf(p.a, p.b); }
__device__ __forceinline__ float add_rows16(float x) { const SwapPair p = swap_rows16(x); return p.a + p.b; }
__device__ __forceinline__ float add_rows32(float x) { const SwapPair p = swap_rows32(x); return p.a + p.b; }
// Within a 16-lane row: value of lane (l - n) mod 16 (DPP row_ror:n).
template <int N>
__device__ __forceinline__ float row_ror(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x120 + N, 0xf, 0xf, false));
}

// Byte offset of the code row of token `t_start` (16-aligned) in the pools,
// for a 16-token sub-tile that lies inside one cache block.
__device__ __forceinline__ size_t subtile_offset(const DecodeArgs &a, int b, int kv, int t_start) {
  const int bs = a.layout.block_size;
  if (a.layout.block_table == nullptr && a.layout.blocks_per_seq == 1)
    return ((static_cast<size_t>(b) * a.num_kv_heads + kv) * bs + t_start) * kL;
  const int blk = t_start / bs;
  const int row = t_start - blk * bs;
  const int logical = b * a.layout.blocks_per_seq + blk;
  const int phys = a.layout.block_table ? a.layout.block_table[logical] : logical;
  return ((static_cast<size_t>(phys) * a.num_kv_heads + kv) * bs + row) * kL;
}

template <int WAVES>
__global__ void __launch_bounds__(WAVES * 64) decode_lut_d128(DecodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[lds_bytes<WAVES>()];
  const uint32_t sbase = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_u8_ptr)smem));
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int split = blockIdx.x % a.n_split;
  const int bk = blockIdx.x / a.n_split;
  const int b = bk / a.num_kv_heads;
  const int kv = bk - b * a.num_kv_heads;
  const int G = a.gqa;

  const int S = a.seq_lens[b];
  const int lo = a.window > 0 ? max(0, S - a.window) : 0;
  const int t0 = max(lo, split * a.chunk);
  const int t1 = min(S, (split + 1) * a.chunk);
  const size_t row0 = static_cast<size_t>(b) * a.num_q_heads + kv * G;

  if (t0 >= t1) {  // nothing attended in this split
    for (int i = tid; i < G * kD; i += WAVES * 64)
      a.part_acc[((row0 + i / kD) * a.n_split + split) * kD + (i % kD)] = 0.f;
    if (tid < G) {
      a.part_ml[2 * ((row0 + tid) * a.n_split + split)] = -INFINITY;
      a.part_ml[2 * ((row0 + tid) * a.n_split + split) + 1] = 0.f;
    }
    return;
  }

  // ---- lane roles
  const int beta = lane >> 4, u = (lane >> 2) & 3, v = lane & 3;
  const int x = 2 * v + (beta & 1);
  uint32_t rsel0 = 0, rsel1 = 0, kc0 = 0, kc1 = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    rsel0 |= static_cast<uint32_t>((k + x) & 7) << (8 * k);
    rsel1 |= static_cast<uint32_t>((k + 4 + x) & 7) << (8 * k);
    kc0 |= static_cast<uint32_t>(64 * u + 8 * ((k + x) & 7)) << (8 * k);
    kc1 |= static_cast<uint32_t>(64 * u + 8 * ((k + 4 + x) & 7)) << (8 * k);
  }
  const uint32_t vbase = sbase + kVBase + 8 * v;

  float m_run = -INFINITY, l_run = 0.f;
  float4_t acc[8];
#pragma unroll
  for (int X = 0; X < 8; ++X) acc[X] = float4_t{0.f, 0.f, 0.f, 0.f};

  const int R0 = t0 & ~63;
  const int nrounds = (t1 - R0 + 63) >> 6;
  const int last16 = (t1 - 1) & ~15;
  const uint8_t *kpool = a.k_codes;
  const uint8_t *vpool = a.v_codes;

  // Code bytes of one round: K windows (bytes 8u..8u+7 of tokens R+16r+4beta+v) and
  // V windows (bytes 8v..8v+7 of tokens R+16u+4beta+s).
  auto load_round = [&](int R, uint2 *kw, uint2 *vw) {
    size_t sub[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) sub[r] = subtile_offset(a, b, kv, min(R + 16 * r, last16));
#pragma unroll
    for (int r = 0; r < 4; ++r)
      kw[r] = *reinterpret_cast<const uint2 *>(kpool + sub[r] + (4 * beta + v) * kL + 8 * u);
    const size_t subu = u == 0 ? sub[0] : (u == 1 ? sub[1] : (u == 2 ? sub[2] : sub[3]));
#pragma unroll
    for (int s = 0; s < 4; ++s)
      vw[s] = *reinterpret_cast<const uint2 *>(vpool + subu + (4 * beta + s) * kL + 8 * v);
  };
  // Two named buffers of code bytes alternate through the token loop (unrolled
  // by two), so no in-flight load destination is ever copied: round rd+W is in
  // flight while round rd is processed.
  uint2 kwA[4], vwA[4], kwB[4], vwB[4];
  if (wave < nrounds) load_round(R0 + 64 * wave, kwA, vwA);

  // ---- setup: value codebook into LDS, table of partial logits via MFMA.
  // All global loads of the setup are issued before any of them is used.
  // Value entry (g, c) goes to kVBase + (g&7)*8192 + 32c + 8(g>>3).
  // Table tile (gb, cb) = groups 4gb..4gb+3 x codes 16cb..16cb+15:
  //   C[(gq,h)][code] = sum_i q'_h[4(4gb+gq)+i] * C_K[4gb+gq][code][i].
  {
    constexpr int NT = WAVES * 64;
    constexpr int VPER = (kL * 256 + NT - 1) / NT;
    const uint2 *vsrc = reinterpret_cast<const uint2 *>(a.cb_v + static_cast<size_t>(kv) * kL * 256 * 4);
    uint2 vst[VPER];
#pragma unroll
    for (int k = 0; k < VPER; ++k) {
      const int e = tid + k * NT;
      if (e < kL * 256) vst[k] = vsrc[e];
    }
    const int m = lane & 15, kq = lane >> 4;
    const int gq = m >> 2, h = m & 3;
    const uint16_t *cbk = a.cb_k + static_cast<size_t>(kv) * kL * 256 * 4;
    const bool lut_wave = wave < kL / 4;        // one group block per wave
    const int gb = wave;
    uint2 kst[16];
    float qv[4] = {0.f, 0.f, 0.f, 0.f};
    if (lut_wave) {
#pragma unroll
      for (int cb = 0; cb < 16; ++cb)
        kst[cb] = *reinterpret_cast<const uint2 *>(
            cbk + (static_cast<size_t>(4 * gb + kq) * 256 + 16 * cb + m) * 4);
      if (kq == gq && h < G) {
        const float4 q4 = *reinterpret_cast<const float4 *>(a.qp + (row0 + h) * kD + 4 * (4 * gb + kq));
        qv[0] = q4.x; qv[1] = q4.y; qv[2] = q4.z; qv[3] = q4.w;
      }
    }
#pragma unroll
    for (int k = 0; k < VPER; ++k) {
      const int e = tid + k * NT;
      if (e < kL * 256) {
        const int g = e >> 8, c = e & 255;
        *reinterpret_cast<uint2 *>(smem + kVBase + (g & 7) * 8192 + (c << 5) + 8 * (g >> 3)) = vst[k];
      }
    }
    if (lut_wave) {
      half4_t a_hi, a_lo;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const _Float16 hi = static_cast<_Float16>(qv[i]);
        a_hi[i] = hi;
        a_lo[i] = static_cast<_Float16>(qv[i] - static_cast<float>(hi));
      }
#pragma unroll
      for (int cb = 0; cb < 16; ++cb) {
        const half4_t bv = __builtin_bit_cast(half4_t, kst[cb]);
        float4_t c = {0.f, 0.f, 0.f, 0.f};
        c = __builtin_amdgcn_mfma_f32_16x16x16f16(a_hi, bv, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x16f16(a_lo, bv, c, 0, 0, 0);
        half4_t o;
        o[0] = static_cast<_Float16>(c[0]);
        o[1] = static_cast<_Float16>(c[1]);
        o[2] = static_cast<_Float16>(c[2]);
        o[3] = static_cast<_Float16>(c[3]);
        // lane (code 16cb+m, group 4gb+kq) holds the 4 heads
        *reinterpret_cast<half4_t *>(smem + (16 * cb + m) * 256 + (4 * gb + kq) * 8) = o;
      }
    }
  }
  __syncthreads();

  auto process_round = [&](const int R, const uint2 *kw, const uint2 *vw) {
    // K: logits of tokens R + 16r + 4beta + u for head v (log2 units); the four
    // sub-tiles are independent chains, interleaved step by step.
    uint32_t w0[4], w1[4];
    float zs[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      w0[r] = __builtin_amdgcn_perm(kw[r].y, kw[r].x, rsel0);
      w1[r] = __builtin_amdgcn_perm(kw[r].y, kw[r].x, rsel1);
      zs[r] = 0.f;
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint32_t sel = 0x0C0C0000u | ((4u + (t & 3)) << 8) | (t & 3);
      half4_t e[4];
#pragma unroll
      for (int r = 0; r < 4; ++r)
        e[r] = tr16_read(sbase + __builtin_amdgcn_perm(t < 4 ? w0[r] : w1[r], t < 4 ? kc0 : kc1, sel));
#pragma unroll
      for (int r = 0; r < 4; ++r) zs[r] = sum4(e[r], zs[r]);
    }
    float z[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tok = R + 16 * r + 4 * beta + u;
      z[r] = (tok >= t0 && tok < t1) ? zs[r] : -INFINITY;
    }

    // online softmax over the round.  Accumulator column (u, v) of the value
    // MFMA mixes the four rows beta, so its reference max is shared by lanes
    // (beta, u, v), beta = 0..3; the four columns u of a head keep their own
    // maxima until the end of the unit.
    float zmax = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
    zmax = max_rows16(zmax);
    zmax = max_rows32(zmax);
    // A column may have no attended token yet (ragged first or last round):
    // then its reference stays -inf and the exponent base is taken as 0.
    const float m_new = fmaxf(m_run, zmax);
    const float m_ref = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_ref);
    float p[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) p[r] = __builtin_amdgcn_exp2f(z[r] - m_ref);
    l_run = l_run * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
    m_run = m_new;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int X = 0; X < 8; ++X) acc[X] *= alpha;
    }
    const half4_t pb = {static_cast<_Float16>(p[0]), static_cast<_Float16>(p[1]),
                        static_cast<_Float16>(p[2]), static_cast<_Float16>(p[3])};
    const half4_t zero4 = {0, 0, 0, 0};

    // V: for token set s (tokens R + 16k + 4beta + s), coordinates of groups 8*(0..3) + X.
    // The eight reads of a set are issued one set ahead of its MFMAs.
    auto v_reads = [&](int s, half4_t *av) {
#pragma unroll
      for (int X = 0; X < 8; ++X) {
        const uint32_t word = X < 4 ? vw[s].x : vw[s].y;
        const uint32_t c = (word >> (8 * (X & 3))) & 0xffu;
        av[X] = tr16_read(vbase + (c << 5) + X * 8192);
      }
    };
    half4_t avA[8], avB[8];
    v_reads(0, avA);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      half4_t *cur = (s & 1) ? avB : avA;
      half4_t *nxt = (s & 1) ? avA : avB;
      if (s < 3) v_reads(s + 1, nxt);
      __builtin_amdgcn_sched_barrier(0);
      const half4_t bset = (u == s) ? pb : zero4;
#pragma unroll
      for (int X = 0; X < 8; ++X)
        acc[X] = __builtin_amdgcn_mfma_f32_16x16x16f16(cur[X], bset, acc[X], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  for (int rd = wave; rd < nrounds; rd += 2 * WAVES) {
    if (rd + WAVES < nrounds) load_round(R0 + 64 * (rd + WAVES), kwB, vwB);
    process_round(R0 + 64 * rd, kwA, vwA);
    if (rd + WAVES >= nrounds) break;
    if (rd + 2 * WAVES < nrounds) load_round(R0 + 64 * (rd + 2 * WAVES), kwA, vwA);
    process_round(R0 + 64 * (rd + WAVES), kwB, vwB);
  }

  // ---- per-wave reduction.  l over the rows of a column; then the four
  // columns u of head v are rescaled to their common max and summed (lanes
  // v, v+4, v+8, v+12 of each row).
  float l_tot = add_rows16(l_run);
  l_tot = add_rows32(l_tot);
  float m_head = fmaxf(m_run, row_ror<4>(m_run));
  m_head = fmaxf(m_head, row_ror<8>(m_head));
  const float wcol = (m_run == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run - m_head);
  l_tot *= wcol;
  l_tot += row_ror<4>(l_tot);
  l_tot += row_ror<8>(l_tot);
#pragma unroll
  for (int X = 0; X < 8; ++X) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float y = acc[X][i] * wcol;
      y += row_ror<4>(y);
      y += row_ror<8>(y);
      acc[X][i] = y;
    }
  }
  m_run = m_head;

  __syncthreads();  // every wave is done with the table before it becomes merge scratch
  float *merge = reinterpret_cast<float *>(smem + kMergeBase);
  float *mw = merge + wave * kMergeFloats;  // [0..4) m, [4..8) l, [8 + h*128 + d) acc
  if (lane < 4) {
    mw[lane] = m_run;
    mw[4 + lane] = l_tot;
  }
  if (u == 0) {
#pragma unroll
    for (int X = 0; X < 8; ++X)
#pragma unroll
      for (int i = 0; i < 4; ++i) mw[8 + v * kD + 32 * beta + 4 * X + i] = acc[X][i];
  }
  __syncthreads();

  // ---- merge the waves and write this split's partials (natural-log max)
  constexpr float kLn2 = 0.693147180559945309f;
  for (int i = tid; i < G * kD; i += WAVES * 64) {
    const int h = i / kD, d = i % kD;
    float big = -INFINITY;
    for (int w = 0; w < WAVES; ++w) big = fmaxf(big, merge[w * kMergeFloats + h]);
    float num = 0.f, den = 0.f;
    if (big != -INFINITY) {
      for (int w = 0; w < WAVES; ++w) {
        const float mwv = merge[w * kMergeFloats + h];
        const float wt = (mwv == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mwv - big);
        num = fmaf(wt, merge[w * kMergeFloats + 8 + h * kD + d], num);
        den = fmaf(wt, merge[w * kMergeFloats + 4 + h], den);
      }
    }
    const size_t r = (row0 + h) * a.n_split + split;
    a.part_acc[r * kD + d] = num;
    if (d == 0) {
      a.part_ml[2 * r] = big == -INFINITY ? -INFINITY : big * kLn2;
      a.part_ml[2 * r + 1] = den;
    }
  }
}

}  // namespace

bool lut_path_eligible(int head_dim, int gqa, int block_size) {
  return head_dim == kD && gqa <= 4 && block_size % 16 == 0;
}

void plan_lut(int batch, int num_kv_heads, int max_seq_len, int *n_split, int *chunk) {
  const long long units = static_cast<long long>(batch) * num_kv_heads;
  int ns = static_cast<int>((256 + units - 1) / units);
  if (ns < 1) ns = 1;
  int ch = (max_seq_len + ns - 1) / ns;
  ch = (ch + 63) & ~63;
  if (ch < 64) ch = 64;
  *chunk = ch;
  *n_split = (max_seq_len + ch - 1) / ch;
}

hipError_t launch_decode_lut(const DecodeArgs &a, hipStream_t stream) {
  constexpr int W = 12;
  const dim3 grid(static_cast<unsigned>(a.batch * a.num_kv_heads * a.n_split));
  decode_lut_d128<W><<<grid, dim3(W * 64), 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace novakv
