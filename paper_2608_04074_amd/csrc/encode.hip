// Append-time encoder: transform new keys/values and store the nearest
// codeword index of every group.
//
// Paper: Algorithm 1 (write step, Q+((k - k_bar) R_K)), Theorem 1 (key
// transform), Corollary 1 (s = v R_V), Sec. "Calibration" (each group gets
// the codeword at the smallest squared distance in the transform domain).
// The transform and the distances are evaluated in fp64 so that the stored
// index is the exact argmin (smallest index among equal distances).
#include <math.h>

#include "encode_block.h"
#include "nova_kv_internal.h"

namespace novakv {

namespace {

// Sink-plus-recent band: a new token's element (bf16 bits) goes to the band
// when its position is there once the append is done (the sequence then ends
// at `end`): a sink slot, or the ring slot of the last n_rec positions.
__device__ __forceinline__ void store_band(const EncodeArgs &a, const int side, const int b, const int kv,
                                           const int pos, const int end, const int d, const uint16_t bits) {
  uint16_t *band = side == 0 ? a.band_k : a.band_v;
  if (!band || !position_in_pool(a.layout, pos)) return;
  if (!(pos < a.n_sink || (a.n_rec > 0 && pos >= end - a.n_rec))) return;
  const int nb = a.n_sink + a.n_rec;
  band[((static_cast<size_t>(b) * a.num_kv_heads + kv) * nb + band_slot(pos, a.n_sink, a.n_rec)) * a.head_dim + d] =
      bits;
}

// bf16 bits of an input element: as stored, or an fp32 value rounded to
// nearest even.
__device__ __forceinline__ uint16_t input_bf16_bits(const EncodeArgs &a, const void *src, const size_t idx) {
  if (a.in_bf16) return static_cast<const uint16_t *>(src)[idx];
  const uint32_t f = __float_as_uint(static_cast<const float *>(src)[idx]);
  return static_cast<uint16_t>((f + 0x7fffu + ((f >> 16) & 1u)) >> 16);
}

// Coordinate q of codeword idx (an index over [Hkv][L][256]): its address,
// the coordinate as loaded from there (the fp16 bits, or the fp8 byte,
// zero-extended), and its value.  Codeword idx + j lies j * 4 elements on.
__device__ __forceinline__ const uint8_t *coordinate_ptr(const void *cb, const bool fp8, const size_t idx, const int q) {
  return static_cast<const uint8_t *>(cb) + (4 * idx + q) * (fp8 ? 1 : 2);
}
__device__ __forceinline__ uint32_t coordinate_raw(const uint8_t *p, const bool fp8, const int j) {
  if (fp8) return p[4 * j];
  return reinterpret_cast<const uint16_t *>(p)[4 * j];
}
__device__ __forceinline__ double coordinate_value(const uint32_t raw, const bool fp8) {
  if (fp8) {
    typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
    const f16x2_t h = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(raw, 1.0f, false);
    return static_cast<double>(static_cast<float>(h[0]));
  }
  return static_cast<double>(half_bits_to_float(static_cast<uint16_t>(raw)));
}

// Cross-lane steps on doubles without LDS traffic (each 32-bit half moves on
// its own).  row_dpp: DPP within 16-lane rows (quad_perm xor 1 = 0xB1, xor 2 =
// 0x4E, row_half_mirror = 0x141, row_mirror = 0x140).  swap_rows: the
// v_permlane{16,32}_swap of x (first operand) and y (second): R = 16
// exchanges the odd rows of x with the even rows of y, R = 32 the high half
// of x with the low half of y; the results are copied out of the returned
// vectors before any reinterpretation.
template <int CTRL>
__device__ __forceinline__ double row_dpp(const double x) {
  const unsigned long long u = static_cast<unsigned long long>(__double_as_longlong(x));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(u), CTRL, 0xf, 0xf, true));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(u >> 32), CTRL, 0xf, 0xf, true));
  return __longlong_as_double(static_cast<long long>((static_cast<unsigned long long>(hi) << 32) | lo));
}
template <int R>
__device__ __forceinline__ void swap_rows(double &x, double &y) {
  static_assert(R == 16 || R == 32, "row distance");
  const unsigned long long ux = static_cast<unsigned long long>(__double_as_longlong(x));
  const unsigned long long uy = static_cast<unsigned long long>(__double_as_longlong(y));
  const uint32_t xl = static_cast<uint32_t>(ux), xh = static_cast<uint32_t>(ux >> 32);
  const uint32_t yl = static_cast<uint32_t>(uy), yh = static_cast<uint32_t>(uy >> 32);
  uint32_t l0, l1, h0, h1;
  if constexpr (R == 16) {
    const auto sl = __builtin_amdgcn_permlane16_swap(xl, yl, false, false);
    const auto sh = __builtin_amdgcn_permlane16_swap(xh, yh, false, false);
    l0 = sl[0], l1 = sl[1], h0 = sh[0], h1 = sh[1];
  } else {
    const auto sl = __builtin_amdgcn_permlane32_swap(xl, yl, false, false);
    const auto sh = __builtin_amdgcn_permlane32_swap(xh, yh, false, false);
    l0 = sl[0], l1 = sl[1], h0 = sh[0], h1 = sh[1];
  }
  x = __longlong_as_double(static_cast<long long>((static_cast<unsigned long long>(h0) << 32) | l0));
  y = __longlong_as_double(static_cast<long long>((static_cast<unsigned long long>(h1) << 32) | l1));
}
// The largest x of the wave, in every lane (swapping x with a copy of itself
// leaves x and the value of lane l ^ R in the two results).
__device__ __forceinline__ double wave_max(double x) {
  x = fmax(x, row_dpp<0xB1>(x));
  x = fmax(x, row_dpp<0x4E>(x));
  x = fmax(x, row_dpp<0x141>(x));
  x = fmax(x, row_dpp<0x140>(x));
  double y = x;
  swap_rows<16>(x, y);
  x = fmax(x, y);
  y = x;
  swap_rows<32>(x, y);
  return fmax(x, y);
}

// Few new tokens per sequence (a decode step): one workgroup per (token,
// sequence, KV head, side, block of 8 groups).  A block needs 32 transform
// columns (D x 32 fp32) and its 8 codebooks (16 KB), so each workgroup
// fetches a quarter (D=128) or half (D=64) of the parameters, all loads
// coalesced and issued before the first use; the launch costs about one
// memory latency.  The block itself is encode_block.h's team computation.
template <int D, bool FP8, bool TBF>
__global__ void __launch_bounds__(256) encode_small(EncodeArgs a) {
  constexpr int L = D / kGroupDim;
  constexpr int NB = L / encblk::kGroups;  // group blocks per token
  __shared__ encblk::Scratch<D> sc;
  const int blk = blockIdx.x % NB;
  const int side = (blockIdx.x / NB) & 1;
  if (side == 1 && a.v_sq) return;  // the scalar value arm has its own kernel
  const int t = blockIdx.x / (2 * NB);
  const int kv = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const void *tm = transform_of(side == 0 ? a.t_k : a.t_v, kv, D, TBF);
  const void *cb = side == 0 ? a.cb_k : a.cb_v;
  const size_t cw0 = static_cast<size_t>(kv) * L * kCodebookSize;
  const void *src = side == 0 ? a.k : a.v;
  uint8_t *pool = side == 0 ? a.k_codes : a.v_codes;
  const int pos = a.start_pos[b] + a.start_offset + t;
  if (!position_in_pool(a.layout, pos)) return;  // uniform: the workgroup stores nothing

  T4 trow[D / 32];
  uint2 cw[encblk::kPer];
  encblk::load_block<D>(tid, tm, TBF, cb, FP8, cw0, blk, trow, cw);
  if (tid < D) {
    const size_t idx = ((static_cast<size_t>(b) * a.n_new + t) * a.num_kv_heads + kv) * D + tid;
    double x = a.in_bf16 ? static_cast<double>(bf16_bits_to_float(static_cast<const uint16_t *>(src)[idx]))
                         : static_cast<double>(static_cast<const float *>(src)[idx]);
    if (side == 0) x -= static_cast<double>(a.kbar[kv * D + tid]);
    sc.xs[tid] = x;
    if (blk == 0 && a.band_k) {
      const int p0 = a.start_pos[b] + a.start_offset;
      store_band(a, side, b, kv, p0 + t, p0 + a.n_new, tid, input_bf16_bits(a, src, idx));
    }
  }
  __syncthreads();
  const size_t off = code_row_offset(a.layout, a.num_kv_heads, L, b, kv, pos);
  int code;
  if (side == 0 && a.k_scales) {
    // Key-scale format: rho needs every coefficient of the key, so the
    // workgroup forms all NB blocks' coefficients (the same computation as
    // the block's own), keeps them in LDS, and searches its block with the
    // coefficients divided by rho; block 0's workgroup stores rho.
    __shared__ double us[D];
    __shared__ double srho;
    T4 tb[D / 32];
    encblk::load_rows<D>(tid, tm, TBF, 0, tb);
    encblk::token_coefficients<D>(tid, sc, tm, TBF, tb, us, [] { __syncthreads(); });
    if (tid == 0) srho = encblk::key_scale<D>(us);
    __syncthreads();
    const double rho = srho;
    double uu[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const double u = us[encblk::kCols * blk + 4 * (tid >> 5) + i];
      uu[i] = rho > 0.0 ? u / rho : 0.0;
    }
    code = encblk::search_codes(tid, uu, cw, FP8);
    if (blk == 0 && tid == 0) a.k_scales[off / L] = encblk::bf16_of(rho);
  } else {
    encblk::partial_block<D>(tid, sc, trow, TBF);
    __syncthreads();
    code = encblk::search_block<D>(tid, sc, cw, FP8);
  }
  if ((tid & 31) == 0) pool[off + encblk::kGroups * blk + (tid >> 5)] = static_cast<uint8_t>(code);
}

// Bulk append: one workgroup (8 waves) per (64-token tile, KV head, sequence,
// side), everything on the fp64 matrix cores.
//  * transform: U = (X - k_bar) T with v_mfma_f64_16x16x4f64 (A = 16 tokens x 4
//    input coordinates from LDS, B = 4 input x 16 output coordinates of T);
//  * distances: per group, rows = codewords, columns = tokens; the accumulator
//    starts at |c|^2 + off_g (off_g >= every |u_g|^2 of the tile, so the value
//    |u - c|^2 + (off_g - |u_g|^2) is >= 0 and ordered like the distance) and
//    the MFMA adds -2 c . u;
//  * argmin: the codeword index replaces the low 8 mantissa bits of the
//    (non-negative) fp64 value, so one min per score keeps the nearest
//    codeword and, on equal values, the smallest index.  The truncation is
//    2^-44 relative, far below the spacing of distinct distances.
// On this part a SIMD does not run VALU work of one wave while it runs
// matrix instructions of another, so the time is the matrix work plus the
// VALU work.  Each wave therefore owns a contiguous run of groups for all
// four 16-token tiles: every codeword tile's conversion and C operand (norms
// from LDS) serve four MFMAs, and the per-group work (norms, offset) is
// shared by 64 tokens.  The codes stay in registers until one store per
// token, and the norms of half a codebook at a time are staged, so the
// workgroup needs 73 KB of LDS and at most 128 VGPRs: two workgroups (four
// waves per SIMD) share a CU.
// LDS rows are padded by two doubles so the operand reads hit distinct banks.
// Operand layout of v_mfma_f64_16x16x4f64 (measured): A[m][k] in lane 16k + m,
// B[k][n] in lane 16k + n, D[m][n] in lane 16 (m mod 4) + n, register m / 4.
constexpr int kBulkWaves = 8;
constexpr int kBulkTokens = 64;

template <int D, bool FP8, bool TBF>
__global__ void __launch_bounds__(64 * kBulkWaves) encode_bulk(EncodeArgs a) {
  constexpr int L = D / kGroupDim;
  constexpr int NW = kBulkWaves;
  constexpr int NT = 64 * NW;            // threads
  constexpr int TT = kBulkTokens;        // tokens per workgroup
  constexpr int NTT = TT / 16;           // token tiles
  constexpr int RS = D + 2;              // LDS row stride (doubles)
  constexpr int OT = D / 16;             // output tiles of the transform
  constexpr int KS = D / 4;              // k-steps of the transform
  constexpr int WPO = NW / OT;           // waves per output tile
  constexpr int TPW = NTT / WPO;         // token tiles per wave in the transform
  constexpr int GPW = L / NW;            // groups per wave in the search
  static_assert(NW % OT == 0 && NTT % WPO == 0 && L % NW == 0, "tiling");
  typedef double double4_t __attribute__((ext_vector_type(4)));
  __shared__ double xs[TT * RS];         // inputs, then coefficients
  __shared__ __attribute__((aligned(32))) double cn[NW][kCodebookSize / 2];  // norms of half a codebook per wave

  const int tile = blockIdx.x, kv = blockIdx.y;
  const int b = blockIdx.z >> 1, side = blockIdx.z & 1;
  if (side == 1 && a.v_sq) return;  // the scalar value arm has its own kernel
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n0 = tile * TT;
  const int nt = min(TT, a.n_new - n0);
  const void *tm = transform_of(side == 0 ? a.t_k : a.t_v, kv, D, TBF);
  const void *cb = side == 0 ? a.cb_k : a.cb_v;
  const size_t cw0 = static_cast<size_t>(kv) * L * kCodebookSize;
  constexpr bool fp8 = FP8;
  const void *src = side == 0 ? a.k : a.v;
  uint8_t *pool = side == 0 ? a.k_codes : a.v_codes;

  // ---- transform operands: wave w computes output tile w mod OT of token
  // tiles tt0 .. tt0 + TPW - 1; its B operands (rows 4ks + q, columns of its
  // tile, of T) are requested first, so that their latency passes while the
  // inputs are staged
  const int m = lane & 15, q = lane >> 4;
  const int ot = wave % OT, tt0 = (wave / OT) * TPW;
  uint32_t tr[KS];  // as loaded (fp32 words, or zero-extended bf16)
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) tr[ks] = load_t1_raw(tm, (4 * ks + q) * D + 16 * ot + m, TBF);

  // inputs (minus k_bar for keys) to LDS in fp64: thread tid stages
  // coordinate tid mod D of tokens tid / D + k * (NT / D)
  static_assert(NT % D == 0, "a thread stages one coordinate");
  {
    constexpr int TP = NT / D, NK = TT / TP;
    const int d = tid % D, t0 = tid / D;
    const double kb = side == 0 ? static_cast<double>(a.kbar[kv * D + d]) : 0.0;
    const size_t row = static_cast<size_t>(a.num_kv_heads) * D;
    const size_t idx0 = ((static_cast<size_t>(b) * a.n_new + n0 + t0) * a.num_kv_heads + kv) * D + d;
    double x[NK];
#pragma unroll
    for (int k = 0; k < NK; ++k) {
      const int t = t0 + k * TP;
      const size_t idx = idx0 + static_cast<size_t>(k * TP) * row;
      x[k] = 0.0;
      if (t < nt)
        x[k] = (a.in_bf16 ? static_cast<double>(bf16_bits_to_float(static_cast<const uint16_t *>(src)[idx]))
                          : static_cast<double>(static_cast<const float *>(src)[idx])) - kb;
    }
#pragma unroll
    for (int k = 0; k < NK; ++k) xs[(t0 + k * TP) * RS + d] = x[k];
    if (a.band_k) {
      const int p0 = a.start_pos[b] + a.start_offset;
      for (int k = 0; k < NK; ++k) {
        const int t = t0 + k * TP;
        if (t < nt)
          store_band(a, side, b, kv, p0 + n0 + t, p0 + a.n_new, d,
                     input_bf16_bits(a, src, idx0 + static_cast<size_t>(k * TP) * row));
      }
    }
  }
  __syncthreads();

  {
    double4_t acc[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) acc[j] = double4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const double bt = static_cast<double>(t1_raw_value(tr[ks], TBF));
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        const double ax = xs[(16 * (tt0 + j) + m) * RS + 4 * ks + q];
        acc[j] = __builtin_amdgcn_mfma_f64_16x16x4f64(ax, bt, acc[j], 0, 0, 0);
      }
    }
    __syncthreads();  // every wave has read its inputs; the coefficients overwrite them
#pragma unroll
    for (int j = 0; j < TPW; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) xs[(16 * (tt0 + j) + 4 * i + q) * RS + 16 * ot + m] = acc[j][i];
  }
  __syncthreads();

  if (side == 0 && a.k_scales) {
    // Key-scale format: rho of each key from its D coefficients, stored as
    // bf16, then the coefficients divided by it (0 when rho = 0).
    double *rhos = &cn[0][0];  // the norms are written only after the last read of these
    if (tid < TT) {
      const double rho = encblk::key_scale<D>(&xs[tid * RS]);
      rhos[tid] = rho;
      const int pos = a.start_pos[b] + a.start_offset + n0 + tid;
      if (tid < nt && position_in_pool(a.layout, pos)) {
        const size_t off = code_row_offset(a.layout, a.num_kv_heads, L, b, kv, pos);
        a.k_scales[off / L] = encblk::bf16_of(rho);
      }
    }
    __syncthreads();
    for (int i = tid; i < TT * D; i += NT) {
      const int t = i / D, d = i % D;
      const double rho = rhos[t];
      xs[t * RS + d] = rho > 0.0 ? xs[t * RS + d] / rho : 0.0;
    }
    __syncthreads();
  }

  // ---- nearest codeword: wave w takes groups GPW*w .. GPW*w + GPW-1 of all
  // token tiles and keeps their codes in registers; the codewords of its next
  // group are requested tile by tile as the current group's are converted
  const int g0 = GPW * wave;
  uint32_t ra[16];  // coordinate q of codeword 16t + m, as loaded
  uint2 rn[4];      // codewords 4 lane .. 4 lane + 3, for their norms
  {
    const size_t cw = cw0 + static_cast<size_t>(g0) * kCodebookSize;
    const uint8_t *cp = coordinate_ptr(cb, fp8, cw + m, q);
#pragma unroll
    for (int t = 0; t < 16; ++t) ra[t] = coordinate_raw(cp, fp8, 16 * t);
#pragma unroll
    for (int j = 0; j < 4; ++j) rn[j] = codeword_raw(cb, fp8, cw + 4 * lane + j);
  }
  uint32_t keep, idx0;
  asm volatile("v_mov_b32 %0, 0xffffff00" : "=v"(keep));
  asm volatile("s_mov_b32 %0, 0" : "=s"(idx0));
  uint32_t code_acc = 0u;  // codes of token lane
  for (int k = 0; k < GPW; ++k) {
    const int g = g0 + k;
    const size_t ncw = cw0 + static_cast<size_t>(min(g + 1, g0 + GPW - 1)) * kCodebookSize;
    const uint8_t *ncp = coordinate_ptr(cb, fp8, ncw + m, q);
    double nc[4], cmax = 0.0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint2 w = codeword_f16(rn[j], fp8);
      const double c0 = half_bits_to_float(static_cast<uint16_t>(w.x & 0xffff));
      const double c1 = half_bits_to_float(static_cast<uint16_t>(w.x >> 16));
      const double c2 = half_bits_to_float(static_cast<uint16_t>(w.y & 0xffff));
      const double c3 = half_bits_to_float(static_cast<uint16_t>(w.y >> 16));
      nc[j] = (c0 * c0 + c1 * c1) + (c2 * c2 + c3 * c3);
      cmax = fmax(cmax, nc[j]);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) rn[j] = codeword_raw(cb, fp8, ncw + 4 * lane + j);
    // offset off_g = M (1 + 2^-39), M the larger of the tile's largest |u_g|^2
    // (lane = token) and the group's largest |c|^2: off_g is at least every
    // |u_g|^2, and the margin off_g - |u_g|^2 >= 2^-39 M exceeds the rounding
    // of a score (a few ulp of a value below 4M)
    double un = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const double u = xs[lane * RS + 4 * g + i];
      un = fma(u, u, un);
    }
    const double big = wave_max(fmax(un, cmax));
    un = big + 0x1p-39 * big;
    // B operands: -2 u (exact scaling), tokens 16 tt + m
    double bu[NTT], best[NTT];
#pragma unroll
    for (int tt = 0; tt < NTT; ++tt) {
      bu[tt] = -2.0 * xs[(16 * tt + m) * RS + 4 * g + q];
      best[tt] = __builtin_huge_val();
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // norms (+ offset) of codewords 128h .. 128h + 127, held by lanes 32h .. 32h + 31
      asm volatile("" ::: "memory");
      if ((lane >> 5) == h) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int c = 4 * (lane & 31) + j;
          cn[wave][16 * (c >> 4) + 4 * (c & 3) + ((c >> 2) & 3)] = nc[j] + un;
        }
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
      __builtin_amdgcn_wave_barrier();
      asm volatile("" ::: "memory");
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int t = 8 * h + s;
        // A operand: coordinate q of codeword 16t + m; the register then
        // receives the next group's codeword
        const double ac = coordinate_value(ra[t], fp8);
        ra[t] = coordinate_raw(ncp, fp8, 16 * t);
        const double4_t cin = *reinterpret_cast<const double4_t *>(&cn[wave][16 * s + 4 * q]);
        double4_t dd[NTT];
#pragma unroll
        for (int tt = 0; tt < NTT; ++tt) dd[tt] = __builtin_amdgcn_mfma_f64_16x16x4f64(ac, bu[tt], cin, 0, 0, 0);
#pragma unroll
        for (int tt = 0; tt < NTT; ++tt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {  // register i = codeword 16t + 4i + q
            const uint32_t idx = idx0 + static_cast<uint32_t>(16 * t + 4 * i);
            const unsigned long long bits = static_cast<unsigned long long>(__double_as_longlong(dd[tt][i]));
            best[tt] = fmin(best[tt], __longlong_as_double(static_cast<long long>(
                                          (bits & 0xffffffff00000000ull) | ((static_cast<uint32_t>(bits) & keep) | idx))));
          }
        // the next tile's MFMAs wait for these minima, so one tile's results
        // are held at a time
#pragma unroll
        for (int tt = 0; tt < NTT; ++tt) asm volatile("" : "+v"(bu[tt]) : "v"(best[tt]));
      }
    }
    // full codeword index 16t + 4i + q into the low byte (q fills its two
    // low bits), then the minimum over the rows q, transposed: rows q and
    // q ^ 1 leave tiles 0 and 2 to the even rows and 1 and 3 to the odd ones,
    // rows q and q ^ 2 tiles 0 and 1 to the low half and 2 and 3 to the high
    // half, so that lane 16q + m ends with tile q's minimum for token m: the
    // code of token lane
    static_assert(NTT == 4, "one token per lane");
#pragma unroll
    for (int tt = 0; tt < NTT; ++tt)
      best[tt] = __longlong_as_double(__double_as_longlong(best[tt]) | static_cast<long long>(q));
    swap_rows<16>(best[0], best[1]);
    swap_rows<16>(best[2], best[3]);
    double lo = fmin(best[0], best[1]), hi = fmin(best[2], best[3]);
    swap_rows<32>(lo, hi);
    const uint32_t code = static_cast<uint32_t>(__double_as_longlong(fmin(lo, hi))) & 0xffu;
    code_acc = (code_acc >> 8) | (code << 24);  // group g0 + k ends in byte 4 - GPW + k
  }
  // the GPW codes of token lane, one store
  if (lane < nt) {
    const int pos = a.start_pos[b] + a.start_offset + n0 + lane;
    if (position_in_pool(a.layout, pos)) {
      uint8_t *row = pool + code_row_offset(a.layout, a.num_kv_heads, L, b, kv, pos) + g0;
      static_assert(GPW == 4 || GPW == 2, "code store width");
      if constexpr (GPW == 4)
        *reinterpret_cast<uint32_t *>(row) = code_acc;
      else
        *reinterpret_cast<uint16_t *>(row) = static_cast<uint16_t>(code_acc >> 16);
    }
  }
}

// Scalar value arm (paper: Sec. "Bit rate" and the implementation table:
// per-token affine INT2 values with a BF16 scale and offset): one workgroup
// (the 256-thread team of encode_block.h) per (new token, KV head,
// sequence).  s = v t_v in fp64 with the block encoder's arithmetic, then
// encode_block.h's levels; coordinate 4g + j goes to bits 2j, 2j + 1 of
// byte g.  The token's value row also goes to the band when it is in it.
template <int D, bool TBF>
__global__ void __launch_bounds__(256) encode_sq_values(EncodeArgs a) {
  constexpr int L = D / kGroupDim;
  __shared__ encblk::Scratch<D> sc;
  __shared__ double us[D];
  __shared__ double red[2 * D / 64];
  __shared__ uint8_t qs[D];
  const int t = blockIdx.x, kv = blockIdx.y, b = blockIdx.z, i = threadIdx.x;
  const int p0 = a.start_pos[b] + a.start_offset;
  if (!position_in_pool(a.layout, p0 + t)) return;  // uniform: the workgroup stores nothing
  const void *tv = transform_of(a.t_v, kv, D, TBF);
  T4 rows[D / 32];
  encblk::load_rows<D>(i, tv, TBF, 0, rows);
  if (i < D) {
    const size_t idx = ((static_cast<size_t>(b) * a.n_new + t) * a.num_kv_heads + kv) * D + i;
    sc.xs[i] = a.in_bf16 ? static_cast<double>(bf16_bits_to_float(static_cast<const uint16_t *>(a.v)[idx]))
                         : static_cast<double>(static_cast<const float *>(a.v)[idx]);
    if (a.band_v) store_band(a, 1, b, kv, p0 + t, p0 + a.n_new, i, input_bf16_bits(a, a.v, idx));
  }
  __syncthreads();
  auto sync = [] { __syncthreads(); };
  encblk::token_coefficients<D>(i, sc, tv, TBF, rows, us, sync);
  uint16_t sb, zb;
  encblk::sq_levels<D>(i, us, red, qs, sync, sb, zb);
  const size_t off = code_row_offset(a.layout, a.num_kv_heads, L, b, kv, p0 + t);
  if (i < L) a.v_codes[off + i] = encblk::sq_byte(qs, i);
  if (i == 0) {
    a.v_sq[(off / L) * 2] = sb;
    a.v_sq[(off / L) * 2 + 1] = zb;
  }
}

// TBF: the transforms are stored as bf16 (a compile-time choice, so that the
// fp32 kernels carry no branch on it).
template <int D, bool TBF>
hipError_t launch_encode_t(const EncodeArgs &a, hipStream_t stream) {
  if (a.v_sq) encode_sq_values<D, TBF><<<dim3(a.n_new, a.num_kv_heads, a.batch), dim3(256), 0, stream>>>(a);
  if (a.n_new <= 4) {
    const dim3 grid(2 * a.n_new * (D / kGroupDim / 8), a.num_kv_heads, a.batch);
    if (a.cb_fp8)
      encode_small<D, true, TBF><<<grid, dim3(256), 0, stream>>>(a);
    else
      encode_small<D, false, TBF><<<grid, dim3(256), 0, stream>>>(a);
  } else {
    const dim3 grid((a.n_new + kBulkTokens - 1) / kBulkTokens, a.num_kv_heads, 2 * a.batch);
    if (a.cb_fp8)
      encode_bulk<D, true, TBF><<<grid, dim3(64 * kBulkWaves), 0, stream>>>(a);
    else
      encode_bulk<D, false, TBF><<<grid, dim3(64 * kBulkWaves), 0, stream>>>(a);
  }
  return hipGetLastError();
}

template <int D>
hipError_t launch_encode_d(const EncodeArgs &a, hipStream_t stream) {
  return a.t_bf16 ? launch_encode_t<D, true>(a, stream) : launch_encode_t<D, false>(a, stream);
}

}  // namespace

hipError_t launch_encode(const EncodeArgs &a, hipStream_t stream) {
  switch (a.head_dim) {
    case 64: return launch_encode_d<64>(a, stream);
    case 128: return launch_encode_d<128>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace novakv
