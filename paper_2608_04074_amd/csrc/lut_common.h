// Device helpers shared by the table-based decode kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace novakv {
namespace lut {

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4_t *lds_short4_ptr;
typedef __attribute__((address_space(3))) uint8_t *lds_u8_ptr;


// Workgroup i of a launch runs on XCD i mod 8.  This maps the launch order to
// a logical order in which each XCD owns one contiguous range: XCD x holds
// logical workgroups [start_x, start_x + count_x), the first n mod 8 XCDs one
// more than the rest.  Consecutive logical workgroups (e.g. the KV heads and
// splits of one sequence) then share an XCD and its L2, and the workgroups
// that read one KV head's parameters spread over all XCDs, so no single L2
// serves every request for the same lines.
__device__ __forceinline__ int xcd_contiguous(const int i, const int n) {
  const int x = i & 7, p = i >> 3;
  const int q = n >> 3, r = n & 7;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + p;
}

// Unit of workgroup number wg in the logical order (split fastest, then
// sequence within a block of b_chunk sequences, then KV head, then sequence
// block).  With the XCD-contiguous remap, an XCD's share of the grid then
// holds all splits of b_chunk sequences for a few KV heads: each KV head's
// parameters are requested by a moderate number of CUs of one L2, and the
// splits of a unit meet in that L2.
__device__ __forceinline__ void unit_of_workgroup(const int wg, const int n_split, const int b_chunk, const int hkv,
                                                  int &kv, int &b, int &split) {
  split = wg % n_split;
  int r = wg / n_split;
  const int bl = r % b_chunk;
  r /= b_chunk;
  kv = r % hkv;
  b = (r / hkv) * b_chunk + bl;
}

__device__ __forceinline__ half4_t tr16_read(uint32_t addr) {
  const short4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4_ptr)(uintptr_t)(addr));
  return __builtin_bit_cast(half4_t, v);
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
// Split partials and arrival counters are exchanged between workgroups that
// may sit on different XCDs, each with its own L2.  Every access to them is a
// relaxed agent-scope atomic (a load or store with device coherence that
// bypasses the non-coherent caches); ordering comes from waiting for these
// stores to complete before the arrival is counted, and from issuing the
// loads only after the last arrival has been observed.  This avoids the L2
// write-back and invalidation that a device-wide fence costs on this part.
__device__ __forceinline__ void store_dev(float *p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_dev(const float *p) {
  return __hip_atomic_load(const_cast<float *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Tagged exchange words.  A published value travels with a tag in the high
// half of one 64-bit word, written and read as a single relaxed agent-scope
// atomic.  The tag is the call's epoch, a nonzero number the host gives
// every decode call: a reader that finds its call's epoch knows that the
// value beside it is the one published in this call, whatever order other
// stores arrived in, so a writer never waits for its stores to complete.
// Words are left in place after use.  A call captured in a graph is
// replayed with its epoch, so there the reader of a slot empties it (zero
// words, tag 0, which no call uses) once its reads are done: each replay
// leaves the exchange all zero and meets no word of the replay before.  The
// host draws odd epochs for direct calls and even ones for captured calls,
// so a replay never takes a word left by a direct call either.
__device__ __forceinline__ void put_word(const uint32_t epoch, uint64_t *p, float v) {
  const uint64_t w = (static_cast<uint64_t>(epoch) << 32) | __builtin_bit_cast(uint32_t, v);
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void clear_word(uint64_t *p) {
  __hip_atomic_store(p, static_cast<uint64_t>(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t get_word(const uint64_t *p) {
  return __hip_atomic_load(const_cast<uint64_t *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool word_ready(const uint32_t epoch, const uint64_t w) {
  return static_cast<uint32_t>(w >> 32) == epoch;
}
__device__ __forceinline__ float word_value(const uint64_t w) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(w));
}

__device__ __forceinline__ float wave_sum(float x) {
  x += row_ror<8>(x);
  x += row_ror<4>(x);
  x += row_ror<2>(x);
  x += row_ror<1>(x);
  return add_rows32(add_rows16(x));
}

}  // namespace lut
}  // namespace novakv
