// Internal declarations shared by the HIP translation units of libnovakv.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "host_checks.h"

namespace novakv {

struct CacheLayout {
  int block_size;
  int blocks_per_seq;
  const int32_t *block_table;  // device [B][blocks_per_seq] or nullptr
};

// Whether position t lies in a sequence's rows of the pools, [0, capacity).
// The encoders store nothing for a position outside it (a step call on an
// empty sequence asks for position -1), as the fused step skips S = 0.
__device__ __forceinline__ bool position_in_pool(const CacheLayout &lay, int t) {
  return t >= 0 && static_cast<long long>(t) < static_cast<long long>(lay.block_size) * lay.blocks_per_seq;
}

// Byte offset of the L code bytes of (sequence b, KV head kv, token t).
__device__ __forceinline__ size_t code_row_offset(const CacheLayout &lay, int num_kv_heads,
                                                  int groups, int b, int kv, int t) {
  const int blk = t / lay.block_size;
  const int row = t - blk * lay.block_size;
  const int logical = b * lay.blocks_per_seq + blk;
  const int phys = lay.block_table ? lay.block_table[logical] : logical;
  return ((static_cast<size_t>(phys) * num_kv_heads + kv) * lay.block_size + row) *
         static_cast<size_t>(groups);
}

struct DecodeArgs {
  int batch, num_q_heads, num_kv_heads, head_dim, gqa;
  const float *kbar;
  const void *t_k_inv_t, *t_v;  // transforms: fp32, or bf16 bit patterns when t_bf16
  int t_bf16;
  const void *cb_k, *cb_v;  // [Hkv][L][256] codewords: 4 fp16, or 4 fp8 E4M3 when cb_fp8
  int cb_fp8;
  CacheLayout layout;
  const void *q;
  int q_bf16;
  const uint8_t *k_codes, *v_codes;
  const uint16_t *k_scales;  // key-scale format: bf16 per-token key scales (pool layout), else nullptr
  const uint16_t *v_sq;      // scalar value arm: bf16 (scale, offset) per token (pool layout), else nullptr
  // Sink-plus-recent band: [B][Hkv][n_sink + n_rec][D] bf16 keys and values
  // of the positions [0, n_sink) and the last n_rec (ring slots), or nullptr
  // (then n_sink = n_rec = 0).
  int n_sink, n_rec;
  const uint16_t *band_k, *band_v;
  const int32_t *seq_lens;
  int max_seq_len, window;
  const float *sinks;
  float scale;      // softmax scale (natural-log units)
  float qscale;     // factor folded into q' (scale, or scale * log2(e) for the table path)
  float *out;
  // workspace carve-out
  int *counters;    // [B][Hkv]       split arrival counters (zero between calls)
  float *qp;        // [B][Hq][D]     pre-transformed, pre-scaled queries
  float *sinkp;     // [B][Hq]        shifted sink logits (-inf when no sink)
  float *part_ml;   // [B][Hq][n_split][2]  running max, denominator
  float *part_acc;  // [B][Hq][n_split][D]  transform-domain value accumulator
  int n_split;      // context splits per sequence
  int chunk;        // tokens per split
  int b_chunk;      // table kernels: sequences per block of the workgroup order (divides batch)
  // Fused step (nova_kv_append_decode_attn): the step's key and value of every
  // sequence are encoded in the launch and stored at position seq_lens[b] - 1.
  // Without a band they are attended from their codes (the pool tokens read
  // are [lo, seq_lens[b] - 1)); with one (n_rec >= 1) the new token is the
  // band's last row, stored there in the launch and attended exactly.
  int append;
  const void *k_new, *v_new;  // [B][Hkv][D]
  int new_bf16;
  const void *t_k;
  uint8_t *k_codes_w, *v_codes_w;  // the pools k_codes / v_codes, written at the new position
  uint16_t *k_scales_w, *v_sq_w;   // the key-scale and scalar-arm pools, written there (else nullptr)
  uint16_t *band_k_w, *band_v_w;   // the band buffers, written at the new token's slot (else nullptr)
  float *newp;      // [B][Hkv][8 items][32] per-block results for the new token
  // Tagged exchange of the head_dim-128 table kernel (64-bit words, the tag
  // in the high half): split partials [B*Hkv][n_split][kXchSlotWords] and
  // the new token's per-block results [B*Hkv][8 items][32].
  uint64_t *xch;
  uint64_t *xnew;
  uint32_t epoch;   // this call's tag of the exchanged words (nonzero, new for every call)
  int clear_xch;    // captured in a graph: readers empty the words they read (replays repeat the epoch)
  // Two-level combine of the head_dim-128 table kernel: splits in groups of
  // group_size, n_group groups (n_group = 1: one level, group_size = n_split);
  // group partials [B*Hkv][n_group][kXchSlotWords]; arrival counters
  // [B*Hkv][1 + n_group] (the groups' count, then one per group).
  int group_size, n_group;
  uint64_t *xgrp;
};

// Words of one split's slot in the exchange: per-head statistics of up to 8
// query heads (16 words), then their accumulators (8 x 64 or 4 x 128
// coordinates).  A second block of the same size holds the split's share of
// the sink-plus-recent band (its own statistics and original-domain
// accumulators).
constexpr int kXchBandWords = 16 + 512;
constexpr int kXchSlotWords = 2 * kXchBandWords;

struct EncodeArgs {
  int batch, n_new, num_kv_heads, head_dim;
  const float *kbar;
  const void *t_k, *t_v;  // transforms: fp32, or bf16 bit patterns when t_bf16
  int t_bf16;
  const void *cb_k, *cb_v;  // [Hkv][L][256] codewords: 4 fp16, or 4 fp8 E4M3 when cb_fp8
  int cb_fp8;
  CacheLayout layout;
  const void *k, *v;
  int in_bf16;
  const int32_t *start_pos;
  int start_offset;  // the first new token of sequence b goes to start_pos[b] + start_offset
  uint8_t *k_codes, *v_codes;
  uint16_t *k_scales;  // key-scale format: bf16 per-token key scales (pool layout), else nullptr
  uint16_t *v_sq;      // scalar value arm: bf16 (scale, offset) per token (pool layout), else nullptr
  int n_sink, n_rec;   // sink-plus-recent band (0, 0 without one)
  uint16_t *band_k, *band_v;
};

constexpr int kMaxBand = 1024;

// Slot of band position p: the sink slots, then a ring of the last n_rec positions.
__host__ __device__ __forceinline__ int band_slot(int p, int n_sink, int n_rec) {
  return p < n_sink ? p : n_sink + p % n_rec;
}

// The attended positions of a sequence of S cached tokens whose range starts
// at lo: sink band [lo, sink_end), codes [code_lo, code_hi), recent band
// [code_hi, S).  Without a band (n_sink = n_rec = 0) everything is codes.
struct AttendedSpans {
  int sink_end, code_lo, code_hi;
};
__host__ __device__ __forceinline__ AttendedSpans attended_spans(int lo, int S, int n_sink, int n_rec) {
  AttendedSpans sp;
  sp.sink_end = lo < n_sink ? (S < n_sink ? S : n_sink) : lo;
  sp.code_lo = lo > n_sink ? lo : n_sink;
  const int r = S - n_rec;
  sp.code_hi = r > sp.code_lo ? r : sp.code_lo;
  if (sp.code_lo > S) sp.code_lo = sp.code_hi = S;
  return sp;
}

// Split plan and workspace carve-out of the decode path.
struct DecodePlan {
  int use_lut;      // 1: table-based stage 1 (decode_lut.hip), 0: generic stage 1
  int n_split;
  int chunk;
  size_t off_cnt, off_qp, off_sinkp, off_ml, off_acc, off_new, off_xch, off_xnew, off_xgrp, total;
};
// Splits tile each sequence's attended span (the last `window` tokens, or all).
// The workspace (off_*, total) is sized for every window and both decode
// paths, so it depends only on (batch, heads, head_dim, max_seq_len);
// block_size <= 0 asks for that size alone.
DecodePlan plan_decode(int batch, int num_q_heads, int num_kv_heads, int head_dim,
                       int max_seq_len, int block_size, int window, bool split_k_only = false);

hipError_t launch_decode(const DecodeArgs &a, int use_lut, hipStream_t stream);
int plan_b_chunk(int batch, int num_kv_heads, int n_split);
// Group size of the two-level combine for n_split splits (n_split when one level suffices).
int plan_group_size(int n_split);

// Table-based decode (head_dim 128 with <= 4, or head_dim 64 with <= 8 query
// heads per KV head; 16-token-aligned blocks): query transform, split pass and
// combine in one launch.
bool lut_path_eligible(int head_dim, int gqa, int block_size);
void plan_lut(int batch, int num_kv_heads, int max_seq_len, int *n_split, int *chunk);
hipError_t launch_decode_lut(const DecodeArgs &a, hipStream_t stream);    // head_dim 128
hipError_t launch_decode_lut64(const DecodeArgs &a, hipStream_t stream);  // head_dim 64
hipError_t launch_encode(const EncodeArgs &a, hipStream_t stream);

__device__ __forceinline__ float half_bits_to_float(uint16_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, h));
}

__device__ __forceinline__ float bf16_bits_to_float(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Four consecutive elements (i a multiple of 4) of a transform (t_k,
// t_k_inv_t, t_v) as loaded, in one load: fp32 words, or with bf16 storage
// two words of bf16 pairs in .x and .y.  They are converted where they are
// used, so that a load issued early is not waited for at its issue.
using T4 = uint4;
__device__ __forceinline__ T4 load_t4(const void *t, const size_t i, const int bf16) {
  if (bf16) {
    const uint2 h = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(t) + i);
    return make_uint4(h.x, h.y, 0u, 0u);
  }
  return *reinterpret_cast<const uint4 *>(static_cast<const float *>(t) + i);
}
__device__ __forceinline__ float4 t4_value(const T4 w, const int bf16) {
  if (bf16)
    return make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u), __uint_as_float(w.y << 16),
                       __uint_as_float(w.y & 0xffff0000u));
  return make_float4(__uint_as_float(w.x), __uint_as_float(w.y), __uint_as_float(w.z), __uint_as_float(w.w));
}
// The [D][D] transform of KV head kv in a [Hkv][D][D] array.
__host__ __device__ __forceinline__ const void *transform_of(const void *t, const int kv, const int D,
                                                             const int bf16) {
  const size_t off = static_cast<size_t>(kv) * D * D;
  return bf16 ? static_cast<const void *>(static_cast<const uint16_t *>(t) + off)
              : static_cast<const void *>(static_cast<const float *>(t) + off);
}
// One element of a transform as loaded (a bf16 element zero-extended), and
// its value.
__device__ __forceinline__ uint32_t load_t1_raw(const void *t, const size_t i, const int bf16) {
  return bf16 ? static_cast<uint32_t>(static_cast<const uint16_t *>(t)[i]) : static_cast<const uint32_t *>(t)[i];
}
__device__ __forceinline__ float t1_raw_value(const uint32_t w, const int bf16) {
  return __uint_as_float(bf16 ? w << 16 : w);
}
// One element of a transform.
__device__ __forceinline__ float t1_value(const void *t, const size_t i, const int bf16) {
  return bf16 ? bf16_bits_to_float(static_cast<const uint16_t *>(t)[i]) : static_cast<const float *>(t)[i];
}

// Raw words of codeword `idx` (an index over [Hkv][L][256]): both words of 4
// fp16, or the 4 fp8 bytes in .x.  One load either way.
__device__ __forceinline__ uint2 codeword_raw(const void *cb, const int fp8, const size_t idx) {
  if (fp8) return make_uint2(static_cast<const uint32_t *>(cb)[idx], 0u);
  return static_cast<const uint2 *>(cb)[idx];
}
// The 4 fp16 coordinates (bit patterns, two per word) of a raw codeword.
// fp8 bytes are OCP E4M3 (sign, 4 exponent bits with bias 7, 3 mantissa
// bits, no infinities); every such value is exact in fp16, and the
// gfx950 conversion with scale 1 gives it exactly, two bytes per instruction.
__device__ __forceinline__ uint2 codeword_f16(const uint2 raw, const int fp8) {
  if (!fp8) return raw;
  typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
  const f16x2_t lo = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(raw.x, 1.0f, false);
  const f16x2_t hi = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(raw.x, 1.0f, true);
  return make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
}
__device__ __forceinline__ uint2 codeword(const void *cb, const int fp8, const size_t idx) {
  return codeword_f16(codeword_raw(cb, fp8, idx), fp8);
}
// Scalar value arm: a code byte's four 2-bit codes (coordinate j in bits
// 2j, 2j+1) as fp16 values 0..3, two per word.
__device__ __forceinline__ uint2 sq_unpack_f16(const uint32_t c) {
  auto h = [](uint32_t q) -> uint32_t { return __builtin_bit_cast(uint16_t, static_cast<_Float16>(q & 3u)); };
  return make_uint2(h(c) | (h(c >> 2) << 16), h(c >> 4) | (h(c >> 6) << 16));
}

// The codebook from codeword idx on (so that later indices stay small).
__device__ __forceinline__ const void *codebook_from(const void *cb, const int fp8, const size_t idx) {
  return fp8 ? static_cast<const void *>(static_cast<const uint32_t *>(cb) + idx)
             : static_cast<const void *>(static_cast<const uint2 *>(cb) + idx);
}

}  // namespace novakv
