// Append-time encoder: transform new keys/values and store the nearest
// codeword index of every group.
//
// Paper: Algorithm 1 (write step, Q+((k - k_bar) R_K)), Theorem 1 (key
// transform), Corollary 1 (s = v R_V), Sec. "Calibration" (exact
// nearest-neighbour search in the Euclidean metric of the transform domain).
// The transform and the distances are evaluated in fp64 so that the stored
// index is the exact argmin (smallest index among equal distances).
#include <math.h>

#include "nova_kv_internal.h"

namespace novakv {

namespace {

constexpr int kThreads = 256;
constexpr int kTokens = 16;  // tokens per workgroup

template <int D>
__global__ void __launch_bounds__(kThreads) encode_v0(EncodeArgs a) {
  constexpr int L = D / kGroupDim;
  constexpr int CB = L * kCodebookSize * kGroupDim;
  __shared__ double xs[kTokens][D];
  __shared__ double us[kTokens][D];
  __shared__ __attribute__((aligned(16))) uint16_t cb[CB];

  const int tile = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int n0 = tile * kTokens;
  const int nt = min(kTokens, a.n_new - n0);
  const int pos0 = a.start_pos[b] + n0;

  for (int side = 0; side < 2; ++side) {
    const float *tm = (side == 0 ? a.t_k : a.t_v) + static_cast<size_t>(kv) * D * D;
    const uint16_t *cbg = (side == 0 ? a.cb_k : a.cb_v) + static_cast<size_t>(kv) * CB;
    const void *src = side == 0 ? a.k : a.v;
    uint8_t *pool = side == 0 ? a.k_codes : a.v_codes;

    {
      const uint4 *s4 = reinterpret_cast<const uint4 *>(cbg);
      uint4 *d4 = reinterpret_cast<uint4 *>(cb);
      for (int i = tid; i < CB * 2 / 16; i += kThreads) d4[i] = s4[i];
    }
    for (int i = tid; i < nt * D; i += kThreads) {
      const int t = i / D, d = i % D;
      const size_t idx =
          ((static_cast<size_t>(b) * a.n_new + n0 + t) * a.num_kv_heads + kv) * D + d;
      double x = a.in_bf16 ? static_cast<double>(bf16_bits_to_float(static_cast<const uint16_t *>(src)[idx]))
                           : static_cast<double>(static_cast<const float *>(src)[idx]);
      if (side == 0) x -= static_cast<double>(a.kbar[kv * D + d]);
      xs[t][d] = x;
    }
    __syncthreads();

    if (tid < D) {
      double acc[kTokens];
#pragma unroll
      for (int t = 0; t < kTokens; ++t) acc[t] = 0.0;
      for (int d = 0; d < D; ++d) {
        const double w = static_cast<double>(tm[d * D + tid]);
#pragma unroll
        for (int t = 0; t < kTokens; ++t) acc[t] = fma(xs[t][d], w, acc[t]);
      }
      for (int t = 0; t < nt; ++t) us[t][tid] = acc[t];
    }
    __syncthreads();

    for (int p = tid; p < nt * L; p += kThreads) {
      const int t = p / L, ell = p % L;
      const double u0 = us[t][ell * 4 + 0], u1 = us[t][ell * 4 + 1];
      const double u2 = us[t][ell * 4 + 2], u3 = us[t][ell * 4 + 3];
      const uint16_t *row = &cb[ell * kCodebookSize * kGroupDim];
      double best = INFINITY;
      int arg = 0;
      for (int c = 0; c < kCodebookSize; ++c) {
#pragma clang fp contract(off)
        const double e0 = u0 - static_cast<double>(half_bits_to_float(row[c * 4 + 0]));
        const double e1 = u1 - static_cast<double>(half_bits_to_float(row[c * 4 + 1]));
        const double e2 = u2 - static_cast<double>(half_bits_to_float(row[c * 4 + 2]));
        const double e3 = u3 - static_cast<double>(half_bits_to_float(row[c * 4 + 3]));
        double dist = e0 * e0;
        dist = dist + e1 * e1;
        dist = dist + e2 * e2;
        dist = dist + e3 * e3;
        if (dist < best) {
          best = dist;
          arg = c;
        }
      }
      const size_t off = code_row_offset(a.layout, a.num_kv_heads, L, b, kv, pos0 + t);
      pool[off + ell] = static_cast<uint8_t>(arg);
    }
    __syncthreads();
  }
}

// Few new tokens per sequence (a decode step): one workgroup per (token,
// sequence, KV head, side).  Every global load (a slice of the transform, the
// lane's codewords) is issued before the first use, so the launch costs about
// one memory latency.  Thread (part, e) forms the part's share of coefficient
// e in fp64; eight lanes (sixteen at D=64) share a group and keep the best
// (distance, index) pair, smallest index on equal distance, before a lane
// reduction.
template <int D>
__global__ void __launch_bounds__(256) encode_small(EncodeArgs a) {
  constexpr int L = D / kGroupDim;
  constexpr int LANES = 256 / L;      // lanes per group (8 at D=128, 16 at D=64)
  constexpr int PER = kCodebookSize / LANES;
  constexpr int PARTS = 256 / D;      // row parts of the transform (2 at D=128, 4 at D=64)
  constexpr int ROWS = D / PARTS;
  __shared__ double xs[D];
  __shared__ double up[PARTS][D];
  __shared__ double us[D];
  const int side = blockIdx.x & 1;
  const int t = blockIdx.x >> 1;
  const int kv = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const float *tm = (side == 0 ? a.t_k : a.t_v) + static_cast<size_t>(kv) * D * D;
  const uint16_t *cbg = (side == 0 ? a.cb_k : a.cb_v) + static_cast<size_t>(kv) * L * kCodebookSize * kGroupDim;
  const void *src = side == 0 ? a.k : a.v;
  uint8_t *pool = side == 0 ? a.k_codes : a.v_codes;
  const int e = tid % D, part = tid / D;
  const int ell = tid / LANES, r = tid % LANES;

  float tcol[ROWS];
#pragma unroll
  for (int j = 0; j < ROWS; ++j) tcol[j] = tm[(part * ROWS + j) * D + e];
  const uint2 *row = reinterpret_cast<const uint2 *>(cbg + static_cast<size_t>(ell) * kCodebookSize * kGroupDim);
  uint2 cw[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) cw[k] = row[r + LANES * k];
  if (tid < D) {
    const size_t idx = ((static_cast<size_t>(b) * a.n_new + t) * a.num_kv_heads + kv) * D + tid;
    double x = a.in_bf16 ? static_cast<double>(bf16_bits_to_float(static_cast<const uint16_t *>(src)[idx]))
                         : static_cast<double>(static_cast<const float *>(src)[idx]);
    if (side == 0) x -= static_cast<double>(a.kbar[kv * D + tid]);
    xs[tid] = x;
  }
  __syncthreads();
  {
    double acc = 0.0;
#pragma unroll
    for (int j = 0; j < ROWS; ++j) acc = fma(xs[part * ROWS + j], static_cast<double>(tcol[j]), acc);
    up[part][e] = acc;
  }
  __syncthreads();
  if (tid < D) {
    double u = up[0][tid];
#pragma unroll
    for (int p = 1; p < PARTS; ++p) u += up[p][tid];
    us[tid] = u;
  }
  __syncthreads();
  const double u0 = us[ell * 4 + 0], u1 = us[ell * 4 + 1], u2 = us[ell * 4 + 2], u3 = us[ell * 4 + 3];
  double best = INFINITY;
  int arg = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
#pragma clang fp contract(off)
    const int c = r + LANES * k;
    const uint2 w = cw[k];
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
  for (int o = LANES / 2; o > 0; o >>= 1) {
    const double ob = __shfl_xor(best, o, 64);
    const int oa = __shfl_xor(arg, o, 64);
    if (ob < best || (ob == best && oa < arg)) {
      best = ob;
      arg = oa;
    }
  }
  if (r == 0) {
    const int pos = a.start_pos[b] + t;
    pool[code_row_offset(a.layout, a.num_kv_heads, L, b, kv, pos) + ell] = static_cast<uint8_t>(arg);
  }
}

template <int D>
hipError_t launch_encode_d(const EncodeArgs &a, hipStream_t stream) {
  if (a.n_new <= 4) {
    const dim3 grid(2 * a.n_new, a.num_kv_heads, a.batch);
    encode_small<D><<<grid, dim3(256), 0, stream>>>(a);
  } else {
    const dim3 grid((a.n_new + kTokens - 1) / kTokens, a.num_kv_heads, a.batch);
    encode_v0<D><<<grid, dim3(kThreads), 0, stream>>>(a);
  }
  return hipGetLastError();
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
