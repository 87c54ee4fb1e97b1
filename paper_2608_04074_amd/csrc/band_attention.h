// Sink-plus-recent band of one (sequence, KV head), computed by the combining
// workgroup of the table-based decode kernels.
//
// Paper: Sec. "Sink-plus-recent band" and the figure of the cache layout at
// decoding position t: the first n_sink and the most recent n_rec positions
// are held in BF16 and attended with their exact keys and values, in the same
// softmax as the positions read from codes.  Their logits carry the same
// shift as the codes' logits, z = (q . k - q . k_bar) * scale (Lemma S1), so
// the band merges with the splits' partials as one more partial; its value
// sum stays in the original domain and is added after the inverse value
// transform.
//
// The band has at most kMaxBand rows per (sequence, KV head) and fits one
// workgroup's LDS:
//  * logits on the matrix cores: 16 band rows per 16x16x32 bf16 MFMA, the
//    query split into a bf16 high part and a bf16 low part (rows h and GM + h
//    of the A operand), so the products carry the query to 2^-17;
//  * per head max and sum of exp(z - max), one wave per head;
//  * values on the VALU in fp32: a lane holds two coordinates of one row;
//  * the rows of a pass (the whole band at the usual sizes) are requested
//    before anything waits for them.
#pragma once

#include "lut_common.h"
#include "nova_kv_internal.h"

namespace novakv {
namespace lut {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

// LDS layout of the band computation (byte offsets in its scratch region).
template <int D, int GM, int VW>
struct BandLds {
  static constexpr uint32_t kQ = 0;                                     // [GM][D] f32 query
  static constexpr uint32_t kStat = kQ + GM * D * 4;                    // m [GM], l [GM]
  static constexpr uint32_t kZ = kStat + 64;                            // [kMaxBand][GM]; then the sum [GM][D]
  static constexpr uint32_t kPart = kZ + kMaxBand * GM * 4;             // [VW][GM][D]; then the scaled output
  static constexpr uint32_t kBytes = kPart + VW * GM * D * 4;
};

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

__device__ __forceinline__ uint16_t bf16_rne(const float x) {
  const uint32_t f = __float_as_uint(x);
  return static_cast<uint16_t>((f + 0x7fffu + ((f >> 16) & 1u)) >> 16);
}

// Attends the G query heads of unit (b, kv) to rows first .. first+count-1
// (count >= 1) of its band positions [lo, sink_end) then [rec_lo, S).  On return, after
// a barrier, the f32 words at kStat hold per head h < G the max of the band
// logits (word h) and the sum of exp(z - max) (word GM + h), and kZ holds the
// value sums acc[h][d] = sum_t exp(z_t - max) v_t[d].  Every thread of the
// workgroup calls it; GM >= G heads, WAVES waves, the first VW of them take
// the values.  q_lds / qk_lds: the query ([GM][D] f32, rows past G unused)
// and q . k_bar per head already in LDS, or nullptr to read q and k_bar here.
template <int D, int GM, int WAVES, int VW>
__device__ __forceinline__ void band_attention(const DecodeArgs &a, uint8_t *scr, const int b, const int kv,
                                               const size_t row0, const int lo, const int sink_end,
                                               const int rec_lo, const int S, const int first, const int count,
                                               const float *q_lds = nullptr, const float *qk_lds = nullptr) {
  using Lay = BandLds<D, GM, VW>;
  static_assert(2 * GM <= 16 && GM % 4 == 0, "the A operand holds the high and low parts of GM heads");
  static_assert(VW <= WAVES && Lay::kBytes <= 65536, "band scratch");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = a.gqa;
  const float *qf = q_lds ? q_lds : reinterpret_cast<const float *>(scr + Lay::kQ);
  float *st = reinterpret_cast<float *>(scr + Lay::kStat);
  float *zb = reinterpret_cast<float *>(scr + Lay::kZ);
  float *part = reinterpret_cast<float *>(scr + Lay::kPart);
  const int ns = sink_end > lo ? sink_end - lo : 0;
  const int nb = count;
  const int nbr = a.n_sink + a.n_rec;
  const size_t hb = (static_cast<size_t>(b) * a.num_kv_heads + kv) * nbr;
  auto row_of = [&](const int i0) -> size_t {
    const int i = first + i0;
    const int p = i < ns ? lo + i : rec_lo + (i - ns);
    return (hb + band_slot(p, a.n_sink, a.n_rec)) * D;
  };

  // Loads are issued a pass at a time, all before their first use: a pass
  // covers 16 KT rows per wave for the keys and TPI VR rows per value wave.
  // The first pass of both is requested before anything else, so the whole
  // band of a usual size (up to 16 KT WAVES rows) costs one memory latency.
  constexpr int KT = 2;
  constexpr int HALF = D / 2, TPI = 64 / HALF;  // value rows per load instruction
  constexpr int VR = 32;
  const int m = lane & 15, kg = lane >> 4;
  const int dp = lane % HALF, ts = lane / HALF;
  const int ntile = (nb + 15) >> 4;
  uint32_t vv[VR];
  auto load_values = [&](const int base) {
#pragma unroll
    for (int j = 0; j < VR; ++j) {
      const int i = base + TPI * (wave + VW * j) + ts;
      vv[j] = (wave < VW && i < nb) ? *reinterpret_cast<const uint32_t *>(a.band_v + row_of(i) + 2 * dp) : 0u;
    }
  };
  bf16x8_t kb[KT][D / 32];
  auto load_keys = [&](const int tbase) {
#pragma unroll
    for (int u = 0; u < KT; ++u) {
      // B column m = band row 16 tile + m (the last row repeats past nb)
      const int i = min(16 * (tbase + wave + WAVES * u) + m, nb - 1);
      const uint16_t *kr = a.band_k + row_of(i);
#pragma unroll
      for (int s = 0; s < D / 32; ++s) kb[u][s] = *reinterpret_cast<const bf16x8_t *>(kr + 32 * s + 8 * kg);
    }
  };
  load_values(0);
  load_keys(0);

  // ---- query in fp32
  if (!q_lds) {
    float *qw = reinterpret_cast<float *>(scr + Lay::kQ);
    for (int i = tid; i < GM * D; i += WAVES * 64) {
      const int h = i / D;
      float x = 0.f;
      if (h < G) {
        const size_t qi = (row0 + h) * D + (i % D);
        x = a.q_bf16 ? bf16_bits_to_float(static_cast<const uint16_t *>(a.q)[qi])
                     : static_cast<const float *>(a.q)[qi];
      }
      qw[i] = x;
    }
    __syncthreads();
  }

  // ---- logits.  Every wave forms q . k_bar of all heads (uniform values) and
  // the A operands: lane (m, kg) holds row m, coordinates 32s + 8kg .. +7.
  float qk[GM];
#pragma unroll
  for (int h = 0; h < GM; ++h) {
    if (qk_lds) {
      qk[h] = qk_lds[h];
    } else {
      float x = 0.f;
#pragma unroll
      for (int j = 0; j < D / 64; ++j)
        x = fmaf(qf[h * D + lane + 64 * j], a.kbar[static_cast<size_t>(kv) * D + lane + 64 * j], x);
      qk[h] = wave_sum(x);
    }
  }
  bf16x8_t aq[D / 32];
#pragma unroll
  for (int s = 0; s < D / 32; ++s) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = m < 2 * GM ? qf[(m % GM) * D + 32 * s + 8 * kg + e] : 0.f;
      const uint16_t hi = bf16_rne(x);
      const uint16_t bits = m < GM ? hi : (m < 2 * GM ? bf16_rne(x - bf16_bits_to_float(hi)) : 0);
      aq[s][e] = __builtin_bit_cast(__bf16, bits);
    }
  }
  for (int tbase = 0; tbase < ntile; tbase += KT * WAVES) {
    if (tbase > 0) load_keys(tbase);
#pragma unroll
    for (int u = 0; u < KT; ++u) {
      const int tt = tbase + wave + WAVES * u;
      float4_t c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < D / 32; ++s) c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq[s], kb[u][s], c, 0, 0, 0);
      // accumulator row r of lane group kg is head 4 kg + r (high parts); the
      // low parts sit 4 GM lanes further
      float zz[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) zz[r] = c[r] + __shfl_down(c[r], 4 * GM, 64);
      const int tok = 16 * tt + m;
      if (tt < ntile && lane < 4 * GM && tok < nb) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int h = 4 * kg + r;
          float qkh = qk[r];
          if constexpr (GM == 8) qkh = kg == 0 ? qk[r] : qk[4 + r];
          zb[tok * GM + h] = h < G ? (zz[r] - qkh) * a.scale : 0.f;  // heads past G: never read
        }
      }
    }
  }
  __syncthreads();

  // ---- per head: max, probabilities, their sum
  if (wave < G) {
    float mx = -INFINITY;
    for (int i = lane; i < nb; i += 64) mx = fmaxf(mx, zb[i * GM + wave]);
    mx = wave_max(mx);
    float l = 0.f;
    for (int i = lane; i < nb; i += 64) {
      const float p = __expf(zb[i * GM + wave] - mx);
      zb[i * GM + wave] = p;
      l += p;
    }
    l = wave_sum(l);
    if (lane == 0) {
      st[wave] = mx;
      st[GM + wave] = l;
    }
  }
  __syncthreads();

  // ---- values: lane (ts, dp) of value wave w takes coordinates 2dp, 2dp + 1
  // of rows base + TPI (w + VW j) + ts
  if (wave < VW) {
    float acc[GM][2];
#pragma unroll
    for (int h = 0; h < GM; ++h) acc[h][0] = acc[h][1] = 0.f;
    for (int base = 0; base < nb; base += TPI * VW * VR) {
      if (base > 0) load_values(base);
#pragma unroll
      for (int j = 0; j < VR; ++j) {
        const int i = base + TPI * (wave + VW * j) + ts;
        if (i < nb) {
          const float v0 = __uint_as_float(vv[j] << 16), v1 = __uint_as_float(vv[j] & 0xffff0000u);
#pragma unroll
          for (int h4 = 0; h4 < GM / 4; ++h4) {
            const float4 p = *reinterpret_cast<const float4 *>(zb + i * GM + 4 * h4);
            acc[4 * h4 + 0][0] = fmaf(p.x, v0, acc[4 * h4 + 0][0]);
            acc[4 * h4 + 0][1] = fmaf(p.x, v1, acc[4 * h4 + 0][1]);
            acc[4 * h4 + 1][0] = fmaf(p.y, v0, acc[4 * h4 + 1][0]);
            acc[4 * h4 + 1][1] = fmaf(p.y, v1, acc[4 * h4 + 1][1]);
            acc[4 * h4 + 2][0] = fmaf(p.z, v0, acc[4 * h4 + 2][0]);
            acc[4 * h4 + 2][1] = fmaf(p.z, v1, acc[4 * h4 + 2][1]);
            acc[4 * h4 + 3][0] = fmaf(p.w, v0, acc[4 * h4 + 3][0]);
            acc[4 * h4 + 3][1] = fmaf(p.w, v1, acc[4 * h4 + 3][1]);
          }
        }
      }
    }
    if constexpr (TPI == 2) {
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        acc[h][0] += __shfl_xor(acc[h][0], 32, 64);
        acc[h][1] += __shfl_xor(acc[h][1], 32, 64);
      }
    }
    if (ts == 0) {
#pragma unroll
      for (int h = 0; h < GM; ++h)
        *reinterpret_cast<float2 *>(part + (wave * GM + h) * D + 2 * dp) = make_float2(acc[h][0], acc[h][1]);
    }
  }
  __syncthreads();
  // ---- sum of the value waves' partials, in wave order (the probabilities are no longer read)
  for (int i = tid; i < GM * D; i += WAVES * 64) {
    float s = 0.f;
    for (int w = 0; w < VW; ++w) s += part[w * GM * D + i];
    zb[i] = s;
  }
  __syncthreads();
}

}  // namespace lut
}  // namespace novakv
