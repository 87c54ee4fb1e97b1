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
constexpr uint32_t kMergeBase = 2 * 65536;  // per-wave merge scratch
constexpr int kMergeFloats = 4 * kD + 8;

template <int WAVES>
constexpr uint32_t lds_bytes() {
  return kMergeBase + WAVES * kMergeFloats * 4;
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

__device__ __forceinline__ float xor_max(float x, int m) { return fmaxf(x, __shfl_xor(x, m, 64)); }
__device__ __forceinline__ float xor_add(float x, int m) { return x + __shfl_xor(x, m, 64); }

// Byte offset of the code row of token `t_start` (16-aligned) in the pools,
// for a 16-token sub-tile that lies inside one cache block.
__device__ __forceinline__ size_t subtile_offset(const DecodeArgs &a, int b, int kv, int t_start) {
  const int bs = a.layout.block_size;
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

  // ---- stage the value codebook: entry (g, c) at kVBase + (g&7)*8192 + 32c + 8(g>>3)
  {
    const uint2 *src = reinterpret_cast<const uint2 *>(a.cb_v + static_cast<size_t>(kv) * kL * 256 * 4);
    for (int e = tid; e < kL * 256; e += WAVES * 64) {
      const int g = e >> 8, c = e & 255;
      *reinterpret_cast<uint2 *>(smem + kVBase + (g & 7) * 8192 + (c << 5) + 8 * (g >> 3)) = src[e];
    }
  }

  // ---- per-query table of partial logits via MFMA:
  // C[(gq,h)][code] = sum_i q'_h[4(4gb+gq)+i] * C_K[4gb+gq][code][i]
  {
    const int m = lane & 15, kq = lane >> 4;
    const int gq = m >> 2, h = m & 3;
    const uint16_t *cbk = a.cb_k + static_cast<size_t>(kv) * kL * 256 * 4;
    for (int gb = wave; gb < kL / 4; gb += WAVES) {
      half4_t a_hi = {0, 0, 0, 0}, a_lo = {0, 0, 0, 0};
      if (kq == gq && h < G) {
        const float *qp = a.qp + (row0 + h) * kD + 4 * (4 * gb + kq);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float xq = qp[i];
          const _Float16 hi = static_cast<_Float16>(xq);
          a_hi[i] = hi;
          a_lo[i] = static_cast<_Float16>(xq - static_cast<float>(hi));
        }
      }
#pragma unroll 4
      for (int cb = 0; cb < 16; ++cb) {
        const uint2 w = *reinterpret_cast<const uint2 *>(
            cbk + (static_cast<size_t>(4 * gb + kq) * 256 + 16 * cb + m) * 4);
        const half4_t bv = __builtin_bit_cast(half4_t, w);
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

  for (int rd = wave; rd < nrounds; rd += WAVES) {
    const int R = R0 + 64 * rd;
    size_t sub[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) sub[r] = subtile_offset(a, b, kv, min(R + 16 * r, last16));
    uint2 kw[4], vw[4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
      kw[r] = *reinterpret_cast<const uint2 *>(kpool + sub[r] + (4 * beta + v) * kL + 8 * u);
    const size_t subu = u == 0 ? sub[0] : (u == 1 ? sub[1] : (u == 2 ? sub[2] : sub[3]));
#pragma unroll
    for (int s = 0; s < 4; ++s)
      vw[s] = *reinterpret_cast<const uint2 *>(vpool + subu + (4 * beta + s) * kL + 8 * v);

    // K: logits of tokens R + 16r + 4beta + u for head v (log2 units)
    float z[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint32_t w0 = __builtin_amdgcn_perm(kw[r].y, kw[r].x, rsel0);
      const uint32_t w1 = __builtin_amdgcn_perm(kw[r].y, kw[r].x, rsel1);
      float zs = 0.f;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint32_t sel = 0x0C0C0000u | ((4u + (t & 3)) << 8) | (t & 3);
        const uint32_t addr = __builtin_amdgcn_perm(t < 4 ? w0 : w1, t < 4 ? kc0 : kc1, sel);
        zs = sum4(tr16_read(sbase + addr), zs);
      }
      const int tok = R + 16 * r + 4 * beta + u;
      z[r] = (tok >= t0 && tok < t1) ? zs : -INFINITY;
    }

    // online softmax over the round (16 lanes share head v)
    float zmax = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
    zmax = xor_max(zmax, 4);
    zmax = xor_max(zmax, 8);
    zmax = xor_max(zmax, 16);
    zmax = xor_max(zmax, 32);
    const float m_new = fmaxf(m_run, zmax);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float p[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) p[r] = __builtin_amdgcn_exp2f(z[r] - m_new);
    l_run = l_run * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
    m_run = m_new;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int X = 0; X < 8; ++X) acc[X] *= alpha;
    }
    const half4_t pb = {static_cast<_Float16>(p[0]), static_cast<_Float16>(p[1]),
                        static_cast<_Float16>(p[2]), static_cast<_Float16>(p[3])};
    const half4_t zero4 = {0, 0, 0, 0};

    // V: for token set s (tokens R + 16k + 4beta + s), coordinates of groups 8*(0..3) + X
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const half4_t bset = (u == s) ? pb : zero4;
#pragma unroll
      for (int X = 0; X < 8; ++X) {
        const uint32_t word = X < 4 ? vw[s].x : vw[s].y;
        const uint32_t c = (word >> (8 * (X & 3))) & 0xffu;
        const half4_t av = tr16_read(vbase + (c << 5) + X * 8192);
        acc[X] = __builtin_amdgcn_mfma_f32_16x16x16f16(av, bset, acc[X], 0, 0, 0);
      }
    }
  }

  // ---- per-wave reduction: sets (lane bits 2,3) for acc; all 16 lanes of a head for l
#pragma unroll
  for (int X = 0; X < 8; ++X) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float y = acc[X][i];
      y = xor_add(y, 4);
      y = xor_add(y, 8);
      acc[X][i] = y;
    }
  }
  float l_tot = xor_add(l_run, 4);
  l_tot = xor_add(l_tot, 8);
  l_tot = xor_add(l_tot, 16);
  l_tot = xor_add(l_tot, 32);

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
  constexpr int W = 8;
  const dim3 grid(static_cast<unsigned>(a.batch * a.num_kv_heads * a.n_split));
  decode_lut_d128<W><<<grid, dim3(W * 64), 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace novakv
