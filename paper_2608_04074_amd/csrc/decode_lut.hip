// Decode attention for head_dim 128 and up to 4 query heads per KV head, in
// one launch: query transform, split pass, and the combine of the splits.
//
// One workgroup owns one (sequence, KV head, context split) unit.  It stages
// the KV head's value codebook in LDS and builds a per-query table of partial
// logits LUT[c][g] = (q'_h[4g..4g+3] . C_K[g][c])_{h<4} (fp16, 64 KB) with
// the 4x4x4 MFMA, so that a key's logit is the sum of its 32 table entries.
// This is the paper's read path (q' = q R_K^{-T} folded in once per step, one
// codebook lookup per group; Sec. "Decoding kernel and read path") with the
// q'-codeword dot products hoisted out of the token loop.
//
// Token loop: waves claim rounds of 64 tokens from an LDS counter and
// prefetch the next round's codes while processing the current one.
//  * K: ds_read_b64_tr_b16 gathers from the table; a 16x16x32 MFMA with a
//    0/1 selector operand sums each token's 32 partials per head.
//  * online softmax in log2 units (q' carries the log2(e) factor), with a
//    lagging reference so the accumulator is rescaled rarely;
//  * V: transposing reads of the staged codebook give the MFMA operand of 8
//    tokens' coordinates; the probabilities (fp16) are the other operand.
// The value accumulator stays in the transform domain (Corollary 1).  Every
// split publishes its partial and counts its arrival; the last one merges
// the partials, adds the sink and applies t_v^T once per head.
//
// The APPEND variant is a whole decode step: it also encodes the step's key
// and value (position seq_len - 1) and merges that token's term after the
// splits, so the cache read covers positions before it only.
#include <math.h>

#include "band_attention.h"
#include "encode_block.h"
#include "lut_common.h"
#include "nova_kv_internal.h"
#include "step_encode.h"

namespace novakv {

namespace {

using namespace lut;

constexpr int kD = 128;
constexpr int kL = kD / kGroupDim;          // 32 groups
constexpr uint32_t kLutBytes = 65536;       // [256 codes][32 groups][4 heads] fp16
constexpr uint32_t kVBase = kLutBytes;      // value codebook, 64 KB
// Per-wave merge scratch: [0..4) m, [4..8) l, then coordinate d of head h at
// 8 + h * kMergeHead + (d / 32) * kMergeBlk + d % 32.  With this padding the 16
// lanes that store a wave's accumulators (one 16-byte store per lane) hit 16
// distinct groups of four banks.
constexpr int kMergeHead = 144, kMergeBlk = 36;
constexpr int kMergeFloats = 8 + 3 * kMergeHead + 3 * kMergeBlk + 32 + 4;
constexpr float kLazyLog2 = 8.f;  // reference lag allowed in the online softmax (log2 units)
// Auxiliary region: query staging (later the combine's s_hat), control words,
// and the fused step's encoder-team counter and per-block results.
constexpr uint32_t kAuxQ = 2 * 65536;              // [4][128] f32
constexpr uint32_t kAuxCtl = kAuxQ + 4 * kD * 4;
// control words: [0] arrival state, [1] next unclaimed round, [4..8) shifted
// sink logits, [8..16) own (m, l) per head
constexpr uint32_t kTeamCtr = kAuxCtl + 64;        // arrivals of the encoder team's waves
constexpr uint32_t kTableCtr = kTeamCtr + 4;       // arrivals of the table waves (two per wave when built)
constexpr uint32_t kItemRes = kTeamCtr + 16;       // [8 items][32] f32
// A region used in turn by the partial sums of q' (setup, [8 parts][4 heads]
// [128] f32), the encoder team's scratch (fused step, early in the loop) and
// the per-wave merge scratch (written by each wave as its loop ends, while
// other waves still read both tables).
constexpr uint32_t kMergeBase = (kItemRes + 8 * 32 * 4 + 255) & ~255u;
constexpr uint32_t kAuxPart = kMergeBase;
// The encoder team's scratch sits past the q' partial sums (16 KiB), so the
// team can encode while the table waves still read those.
constexpr uint32_t kAppendScratch = kMergeBase + 16384;
constexpr uint32_t kLdsBytes = kMergeBase + 12 * kMergeFloats * 4;
// Once every wave has left the loop, the value-codebook region holds the
// split's own merged partial ([4][128] at kAuxOwn) and the combine's partial
// outputs.
constexpr uint32_t kAuxOwn = kVBase;
constexpr uint32_t kAuxOut = kVBase + 4 * kD * 4;
static_assert(32 * kD * 4 <= 16384 && 16384 + sizeof(step::Scratch<kD>) <= 12 * kMergeFloats * 4 &&
                  16384 + 2 * sizeof(encblk::Scratch<kD>) <= 12 * kMergeFloats * 4,
              "the q' partial sums and, past them, the encoder team's scratch fit in the merge region");
static_assert(kLdsBytes <= 160 * 1024, "LDS budget of a workgroup");
constexpr float kLn2 = 0.693147180559945309f;

template <int WAVES, bool APPEND>
constexpr uint32_t lds_bytes() {
  static_assert(WAVES == 12, "the merge region holds 12 waves' scratch; waves 8..11 form the sink logits");
  return kLdsBytes;
}


// Byte offset of the code row of token `t_start` (16-aligned) in the pools,
// for a 16-token sub-tile that lies inside one cache block.
// bs_shift = log2(block_size) when it is a power of two, else -1.
__device__ __forceinline__ size_t subtile_offset(const DecodeArgs &a, int b, int kv, int t_start, int bs_shift) {
  const int bs = a.layout.block_size;
  if (a.layout.block_table == nullptr && a.layout.blocks_per_seq == 1)
    return ((static_cast<size_t>(b) * a.num_kv_heads + kv) * bs + t_start) * kL;
  const int blk = bs_shift >= 0 ? (t_start >> bs_shift) : t_start / bs;
  const int row = t_start - blk * bs;
  const int logical = b * a.layout.blocks_per_seq + blk;
  const int phys = a.layout.block_table ? a.layout.block_table[logical] : logical;
  return ((static_cast<size_t>(phys) * a.num_kv_heads + kv) * bs + row) * kL;
}

// Work of one (sequence, KV head, split) unit that attends to at least one
// token: q' of the unit's query heads, the two LDS tables, the token loop, and
// the split's partials (max in natural-log units, denominator, accumulator).
// Thread t < 512 of a workgroup holds row (t mod 128) of t_v, columns
// 32 * (t / 128) .. +31, for the inverse value transform of the combine.
template <bool TBF>
__device__ __forceinline__ void load_tv_rows(const DecodeArgs &a, const int kv, T4 (&tv)[8]) {
  const int tid = threadIdx.x;
  if (tid < 512) {
    const size_t row = (static_cast<size_t>(kv) * kD + (tid & (kD - 1))) * kD + 32 * (tid >> 7);
#pragma unroll
    for (int i = 0; i < 8; ++i) tv[i] = load_t4(a.t_v, row + 4 * i, TBF);
  }
}

// Exchange between the splits of a (sequence, KV head).  Each split's merge
// threads publish its partial as tagged words as they form it, and the
// encoder team publishes the new token's blocks as it computes them, without
// waiting for the stores to land; thread kCtl, alone in its wave so that no
// other memory operation of that wave delays its reply (a wave's memory
// operations complete in issue order), counts the split in while the waves
// merge.  The split that brings the count to n_split combines: it checks the
// tag of every word it reads (the call's epoch), so no order between the
// stores and the count is needed.  In a call captured in a graph, whose
// replays repeat its epoch, it then empties every word of the unit's slots
// and new-token blocks, its own included, so each replay leaves the exchange
// all zero.  With many splits the count runs per group of splits, and the
// group's last split merges the group first (two levels, below).
//   split slot: log-sum-exp m + ln l of head h at word 2h (natural log),
//               normalised coordinate d of head h (acc / l) at 2G + h*128 + d;
//               a split without tokens publishes nothing;
//   new token:  item k (side * 4 + block), lane j at word 32k + j, key
//               blocks for lanes j < G (the heads), value blocks for all 32.
constexpr int kCtl = 512;
// Bound of the wait for a word whose writer has already counted itself in:
// it only has to complete a store, so the bound is never reached in practice.
constexpr int kSpinLimit = 1 << 20;

// Fused step: this split's share of the new token's encode.  Item i =
// side * 4 + block (blocks of 8 groups) is done by split i mod n_eff.  Waves
// 8..11 (the encoder team, 256 threads) take this split's items one after the
// other with the shared block encoder (encode_block.h), from the end of the
// value-codebook staging, while waves 0..7 build the tables and then start
// the token loop (rounds are claimed dynamically, so the team's waves simply
// take fewer).  The team synchronises through an LDS arrival counter instead
// of workgroup barriers, and waits on the table waves' counter before it
// reads the tables.  Each item
// stores its codes at position p of the pools and leaves its contribution in
// LDS: a key block the partial logits of its 8 groups for each head (table
// entries of the stored codes, added in group order), a value block its 32
// coordinates of the decoded value (transform domain).
__device__ __forceinline__ int items_of_split(const int split, const int n_eff) {
  return (8 - split + n_eff - 1) / n_eff;  // items split, split + n_eff, ... below 8
}

// All four waves of the team arrive, then each continues once the counter
// has reached 4 * phase: LDS writes before the call are visible after it.
__device__ __forceinline__ void team_sync(uint8_t *smem, const int phase) {
  step::team_meet(reinterpret_cast<int *>(smem + kTeamCtr), phase);
}

// The eight table waves arrive, then each continues once all eight have
// (8 * phase arrivals): LDS writes before the call are visible after it.
__device__ __forceinline__ void table_meet(int *ctr, const int phase) {
  if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
  while (__hip_atomic_load(ctr, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < 8 * phase)
    __builtin_amdgcn_s_sleep(1);
}

// The loads of the team's k-th item (thread t = tid - 512 of the team).
struct ItemRegs {
  T4 trow[kD / 32];
  uint2 cw[encblk::kPer];
  double x;  // thread t < D: element t of the token minus k_bar (keys) or of the token (values)
};

// The transform columns and the token element of the item (its rows).
template <bool TBF>
__device__ __forceinline__ void load_item_rows(const DecodeArgs &a, const int b, const int kv, const int split,
                                               const int n_eff, const int k, const int t, ItemRegs &r) {
  const int item = split + k * n_eff;
  const int side = item >> 2, blk = item & 3;
  encblk::load_rows<kD>(t, transform_of(side == 0 ? a.t_k : a.t_v, kv, kD, TBF), TBF, blk, r.trow);
  if (t < kD) {
    const void *src = side == 0 ? a.k_new : a.v_new;
    const size_t idx = (static_cast<size_t>(b) * a.num_kv_heads + kv) * kD + t;
    double x = a.new_bf16 ? static_cast<double>(bf16_bits_to_float(static_cast<const uint16_t *>(src)[idx]))
                          : static_cast<double>(static_cast<const float *>(src)[idx]);
    if (side == 0) x -= static_cast<double>(a.kbar[kv * kD + t]);
    r.x = x;
  }
}

// The codewords of the item's 8 groups.
// (fp8: the codebook format, a compile-time constant at every call)
__device__ __forceinline__ void load_item_cw(const DecodeArgs &a, const int kv, const int split, const int n_eff,
                                             const int k, const int t, ItemRegs &r, const bool fp8) {
  const int item = split + k * n_eff;
  const int side = item >> 2, blk = item & 3;
  encblk::load_codewords(t, side == 0 ? a.cb_k : a.cb_v, fp8, static_cast<size_t>(kv) * kL * 256, blk, r.cw);
}

template <bool TBF>
__device__ __forceinline__ void load_item(const DecodeArgs &a, const int b, const int kv, const int split,
                                          const int n_eff, const int k, const int t, ItemRegs &r, const bool fp8) {
  load_item_rows<TBF>(a, b, kv, split, n_eff, k, t, r);
  load_item_cw(a, kv, split, n_eff, k, t, r, fp8);
}

// Team meetings of the encode: two per item (its x in LDS, then the wave
// partials) and one after the last item, before the key blocks' head sums.
__device__ __forceinline__ int team_phases(const int split, const int n_eff) {
  return 2 * items_of_split(split, n_eff) + 1;
}

// Called by the team's threads only (t = tid - 512) while the table waves
// build the tables (the key blocks wait for them, counter tctr, before their
// table lookups).  Each item requests its loads when it starts.  Items
// alternate between two scratch areas, so no meeting guards their reuse.  The
// thread that found a group's codeword records its per-group result: a key
// block's partial logits of the 8 groups per head (table entries of the
// stored codes, res[32 k + 4 gg + h]), a value block's coordinates
// (res[32 k + 4 gg + i]).  After the last item thread h < G of the team sums
// each key block's head h over the groups in order, into res[32 k + h].
template <bool TBF>
__device__ __forceinline__ void encode_items(const DecodeArgs &a, uint8_t *smem, const int b, const int kv,
                                             const int split, const int n_eff, const size_t tokoff, const int t,
                                             const bool fp8, int *tctr) {
  encblk::Scratch<kD> *sc = reinterpret_cast<encblk::Scratch<kD> *>(smem + kAppendScratch);  // [2]
  float *res = reinterpret_cast<float *>(smem + kItemRes);
  uint64_t *xn = a.xnew + static_cast<size_t>(b * a.num_kv_heads + kv) * 8 * 32;
  const int G = a.gqa;
  const int nmine = items_of_split(split, n_eff);
  int phase = 0;
  auto encode_one = [&](const int k, const ItemRegs &ri) {
    const int item = split + k * n_eff;
    const int side = item >> 2, blk = item & 3;
    encblk::Scratch<kD> &s = sc[k & 1];
    if (t < kD) s.xs[t] = ri.x;
    team_sync(smem, ++phase);
    encblk::partial_block<kD>(t, s, ri.trow, TBF);
    team_sync(smem, ++phase);
    const int code = encblk::search_block<kD>(t, s, ri.cw, fp8);
    const int gl = t >> 5, lr = t & 31;
    const int g = encblk::kGroups * blk + gl;
    if (lr == 0) (side == 0 ? a.k_codes_w : a.v_codes_w)[tokoff + g] = static_cast<uint8_t>(code);
    if (lr < 4) {
      float v;
      if (side == 0) {
        // the key tables: built by the table waves meanwhile
        while (__hip_atomic_load(tctr, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < 16)
          __builtin_amdgcn_s_sleep(1);
        v = lr < G ? static_cast<float>(*reinterpret_cast<const _Float16 *>(smem + code * 256 + g * 8 + 2 * lr)) : 0.f;
      } else {
        v = static_cast<float>(*reinterpret_cast<const _Float16 *>(smem + kVBase + (g & 7) * 8192 + 32 * code +
                                                                   8 * (g >> 3) + 2 * lr));
        if (a.n_split > 1) put_word(a.epoch, xn + item * 32 + 4 * gl + lr, v);
      }
      res[item * 32 + 4 * gl + lr] = v;
    }
  };
  for (int k = 0; k < nmine; ++k) {
    ItemRegs r;
    load_item<TBF>(a, b, kv, split, n_eff, k, t, r, fp8);
    encode_one(k, r);
  }
  team_sync(smem, ++phase);
  if (t < G) {
    for (int item = split; item < 4; item += n_eff) {
      float v = 0.f;
#pragma unroll
      for (int gg = 0; gg < encblk::kGroups; ++gg) v += res[item * 32 + 4 * gg + t];
      res[item * 32 + t] = v;
      if (a.n_split > 1) put_word(a.epoch, xn + item * 32 + t, v);
    }
  }
}

// BSTEP: a fused step with a band (APPEND too): the new token is the band's
// last row, and the team runs step::encode_token (step_encode.h): task j of
// the new token's encode goes to split j mod n_eff.
template <int WAVES, bool APPEND, bool KS, bool FP8, bool SQ, bool BSTEP, bool TBF>
__device__ __forceinline__ void split_pass(const DecodeArgs &a, uint8_t *smem, const int b, const int kv,
                                           const int split, const int t0, const int t1, const size_t row0,
                                           const int rot, const int n_eff, const int S, T4 (&tv)[8]) {
  const uint32_t sbase = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_u8_ptr)smem));
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = a.gqa;

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
  float z_run = 0.f;  // scalar value arm: sum of p * offset of the column's tokens
  float4_t acc[8];
#pragma unroll
  for (int X = 0; X < 8; ++X) acc[X] = float4_t{0.f, 0.f, 0.f, 0.f};

  // A split with no token of its own (t1 == t0) runs the setup and an empty
  // loop: its round requests read row 0 of physical block 0, which every
  // pool has, instead of positions of its sequence.
  const bool act = t1 > t0;
  const int R0 = t0 & ~63;
  const int nrounds = act ? (t1 - R0 + 63) >> 6 : 0;
  const int last16 = max(0, (t1 - 1) & ~15);
  const uint8_t *kpool = a.k_codes;
  const uint8_t *vpool = a.v_codes;

  // Code bytes of one round: K windows (bytes 8u..8u+7 of tokens R+16r+4beta+v) and
  // V windows (bytes 8v..8v+7 of tokens R+16beta+4u+s).
  const int bsz = a.layout.block_size;
  const int bs_shift = (bsz & (bsz - 1)) == 0 ? __builtin_ctz(bsz) : -1;
  const uint32_t koff = (4 * beta + v) * kL + 8 * u;  // lane offsets inside a 16-token sub-tile
  const uint32_t voff = 4 * u * kL + 8 * v;
  // Key-scale format: lane (beta, j) also loads the stored scale of token
  // j of sub-tile beta, issued after the code bytes; the scalar value arm
  // loads that token's (scale, offset) word the same way.
  auto load_round = [&](int R, uint2 *kw, uint2 *vw, uint32_t &ks, uint32_t &vq) {
    size_t sub[4];  // uniform: byte offsets of the round's four sub-tiles
#pragma unroll
    for (int r = 0; r < 4; ++r)
      sub[r] = act ? subtile_offset(a, b, kv, min(R + 16 * r, last16), bs_shift) : static_cast<size_t>(kv) * bsz * kL;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint8_t *kb = kpool + sub[r];
      kw[r] = *reinterpret_cast<const uint2 *>(kb + koff);
    }
    const size_t subb = beta == 0 ? sub[0] : (beta == 1 ? sub[1] : (beta == 2 ? sub[2] : sub[3]));
    const uint8_t *vb = vpool + subb;
#pragma unroll
    for (int s = 0; s < 4; ++s) vw[s] = *reinterpret_cast<const uint2 *>(vb + voff + s * kL);
    if constexpr (KS) ks = a.k_scales[subb / kL + (lane & 15)];
    if constexpr (SQ) vq = reinterpret_cast<const uint32_t *>(a.v_sq)[subb / kL + (lane & 15)];
  };
  // Two named buffers of code bytes alternate through the token loop (unrolled
  // by two), so no in-flight load destination is ever copied: round rd+W is in
  // flight while round rd is processed.
  // Two round buffers: wave w requests round w during the setup; afterwards
  // each wave claims its next round from a workgroup counter when it starts
  // processing the current one, so waves that the issue arbiter serves less
  // often simply take fewer rounds and all waves end together.
  uint2 kwb[2][4], vwb[2][4];
  uint32_t ksb[2] = {0u, 0u}, vqb[2] = {0u, 0u};
  int *rctr = reinterpret_cast<int *>(smem + kAuxCtl) + 1;
  if (tid == 0) {
    *rctr = WAVES;  // rounds 0 .. WAVES-1 are taken; visible after the setup's barrier
    *reinterpret_cast<int *>(smem + kTableCtr) = 0;
    if constexpr (APPEND) *reinterpret_cast<int *>(smem + kTeamCtr) = 0;
  }

  // ---- setup: value codebook into LDS, table of partial logits via MFMA.
  // All global loads of the setup are issued before any of them is used, in
  // the order query, t_k_inv_t rows, key codebook, value codebook, k_bar,
  // first round of codes.  A wave's loads complete in issue order and the
  // compiler's waits assume the fewest loads any path issued, so everything
  // younger than the value codebook is issued by every wave: the staging then
  // waits for nothing past the codebook, and the first round's HBM reads stay
  // in flight through the setup.
  // Value entry (g, c) goes to kVBase + (g&7)*8192 + 32c + 8(g>>3); element e
  // of the staging pass maps to (g, c) so that the 32 lanes of a half-wave
  // write 32 distinct bank pairs.
  // Table: the 16-block 4x4x4 MFMA gives every 4-lane block its own group, so
  // one instruction produces 16 groups x 4 codes x 4 heads:
  //   LUT[c][g][h] = sum_i q'_h[4g+i] * C_K[g][c][i].
  {
    constexpr int NT = WAVES * 64;
    // q' = q t_k_inv_t (Theorem 1: the query side of the key transform),
    // formed here for the unit's query heads.  Thread (jq, e4) < 512 holds
    // rows 8*jq .. 8*jq+7 of columns 4*e4 .. 4*e4+3.
    const int e4 = tid & 31, jq = tid >> 5;
    // thread t < 512 stages element t & 127 of head t >> 7 (heads past G repeat
    // head G-1 and are never used): one 32-bit load of the word holding it,
    // converted only when it is stored
    const size_t qi = (row0 + min(tid >> 7, G - 1)) * kD + (tid & (kD - 1));
    uint32_t qword = 0;
    T4 trow[8];
    if (tid < 512) {
      qword = a.q_bf16 ? reinterpret_cast<const uint32_t *>(a.q)[qi >> 1] : reinterpret_cast<const uint32_t *>(a.q)[qi];
      const size_t tk = (static_cast<size_t>(kv) * kD + 8 * jq) * kD + 4 * e4;
#pragma unroll
      for (int r = 0; r < 8; ++r) trow[r] = load_t4(a.t_k_inv_t, tk + r * kD, TBF);
    }
    // table waves: group set (wave & 1) of 16 groups, code range 64*(wave >> 1) .. +63
    const bool lut_wave = wave < 8;
    const int lg = 16 * (wave & 1) + (lane >> 2);  // this lane's group
    const int lj = lane & 3;                       // head (A operand) / code in a quad (B, D)
    const int cbase = 64 * (wave >> 1);
    // codewords as raw words (fp16, or fp8 bytes converted where they are used)
    constexpr bool fp8 = FP8;
    const void *cbk = codebook_from(a.cb_k, fp8, static_cast<size_t>(kv) * kL * 256);
    const void *cbv = codebook_from(a.cb_v, fp8, static_cast<size_t>(kv) * kL * 256);
    uint2 kst[16];
    if (lut_wave) {
#pragma unroll
      for (int t = 0; t < 16; ++t) kst[t] = codeword_raw(cbk, fp8, lg * 256 + cbase + 4 * ((t + rot) & 15) + lj);
    }
    constexpr int VPER = (kL * 256 + NT - 1) / NT;
    auto vmap = [](int e, int &g, int &c) {
      const int r = e >> 5;
      g = 8 * ((e >> 3) & 3) + (r & 7);
      c = 8 * (r >> 3) + (e & 7);
    };
    // the workgroups that share a KV head start at different offsets, so their
    // simultaneous requests for the same parameters spread over the L2 channels
    const int vrot = 256 * (rot & 31);
    // elements past the codebook wrap onto entries that other threads also
    // stage: the same value is written twice
    uint2 vst[VPER];
    if constexpr (!SQ) {
#pragma unroll
      for (int k = 0; k < VPER; ++k) {
        int g, c;
        vmap((tid + k * NT + vrot) & (kL * 256 - 1), g, c);
        vst[k] = codeword_raw(cbv, fp8, g * 256 + c);
      }
    }
    // waves 8 .. 8+G-1 form the shifted sink logit of head wave-8 (Lemma S1)
    const int sh = wave - 8;
    const float2 kb2 = *reinterpret_cast<const float2 *>(a.kbar + static_cast<size_t>(kv) * kD + 2 * lane);
    // a wave without a round of its own (nrounds >= 1 in an active split)
    // re-reads the last round and never processes it
    load_round(max(0, R0 + 64 * min(wave, nrounds - 1)), kwb[0], vwb[0], ksb[0], vqb[0]);
    float *qs = reinterpret_cast<float *>(smem + kAuxQ);       // [4][128] query
    // partial q': [8 parts][32 groups][4 heads][4 coordinates], so that a table
    // lane's float4 (its group, its head) sits next to its neighbours'
    float *qsum = reinterpret_cast<float *>(smem + kAuxPart);
    if (tid < 512) {
      const uint32_t qb = a.q_bf16 ? ((qi & 1) ? (qword & 0xffff0000u) : (qword << 16)) : qword;
      qs[tid] = __uint_as_float(qb);
    }
#pragma unroll
    for (int k = 0; k < VPER; ++k) {
      int g, c;
      vmap((tid + k * NT + vrot) & (kL * 256 - 1), g, c);
      // scalar value arm: every group's table maps a code byte to its four
      // 2-bit codes q (0..3, exact in fp16), so the value MFMA sums
      // p * scale * q; the offsets are summed apart
      const uint2 e = SQ ? sq_unpack_f16(c) : codeword_f16(vst[k], fp8);
      *reinterpret_cast<uint2 *>(smem + kVBase + (g & 7) * 8192 + (c << 5) + 8 * (g >> 3)) = e;
    }
    __syncthreads();
    // The sink logits (waves 8 .. 8+G-1), the partial sums of q' (waves
    // 0..7) and the tables (waves 0..7).
    auto sink_logits = [&] {
      if (sh < G) {
        const float dot = wave_sum(fmaf(qs[sh * kD + 2 * lane], kb2.x, qs[sh * kD + 2 * lane + 1] * kb2.y));
        if (lane == 0) {
          reinterpret_cast<float *>(smem + kAuxCtl)[4 + sh] = a.sinks ? a.sinks[kv * G + sh] - a.scale * dot : -INFINITY;
          // q . k_bar itself for the band's logits (a fused step without a band
          // keeps its encoder results in this region)
          if constexpr (!APPEND || BSTEP) reinterpret_cast<float *>(smem + kItemRes)[sh] = dot;
        }
      }
    };
    auto q_partials = [&] {
      {  // tid < 512
        float4 acc[4];
#pragma unroll
        for (int hh = 0; hh < 4; ++hh) {
          acc[hh] = make_float4(0.f, 0.f, 0.f, 0.f);
          const float4 q0 = *reinterpret_cast<const float4 *>(qs + hh * kD + 8 * jq);
          const float4 q1 = *reinterpret_cast<const float4 *>(qs + hh * kD + 8 * jq + 4);
          const float qq[8] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w};
#pragma unroll
          for (int r = 0; r < 8; ++r) {
            const float4 tr = t4_value(trow[r], TBF);
            acc[hh].x = fmaf(qq[r], tr.x, acc[hh].x);
            acc[hh].y = fmaf(qq[r], tr.y, acc[hh].y);
            acc[hh].z = fmaf(qq[r], tr.z, acc[hh].z);
            acc[hh].w = fmaf(qq[r], tr.w, acc[hh].w);
          }
        }
        // lanes l and l + 32 hold rows of the same columns: fold them, one part per wave
#pragma unroll
        for (int hh = 0; hh < 4; ++hh) {
          acc[hh].x = add_rows32(acc[hh].x);
          acc[hh].y = add_rows32(acc[hh].y);
          acc[hh].z = add_rows32(acc[hh].z);
          acc[hh].w = add_rows32(acc[hh].w);
          if (lane < 32) *reinterpret_cast<float4 *>(qsum + wave * 512 + e4 * 16 + hh * 4) = acc[hh];
        }
      }
    };
    auto build_tables = [&] {
      {  // a table wave
        float qv[4] = {0.f, 0.f, 0.f, 0.f};
        if (lj < G) {
#pragma unroll
          for (int pp = 0; pp < 8; ++pp) {
            const float4 x4 = *reinterpret_cast<const float4 *>(qsum + pp * 512 + lg * 16 + lj * 4);
            qv[0] += x4.x; qv[1] += x4.y; qv[2] += x4.z; qv[3] += x4.w;
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) qv[i] *= a.qscale;
        }
        half4_t a_hi, a_lo;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const _Float16 hi = static_cast<_Float16>(qv[i]);
          a_hi[i] = hi;
          a_lo[i] = static_cast<_Float16>(qv[i] - static_cast<float>(hi));
        }
        // After the MFMA of step t, lane 4b + j holds the 4 heads of (group
        // 16*(wave&1) + b, code cbase + 4*((t + rot) & 15) + j); all 4 lanes of a
        // block hit the bank pair of their group.  Two steps are exchanged across
        // the wave halves first, so that each half-wave writes 16 groups x 2
        // codes (2 lanes per bank pair instead of 4): lanes j < 2 keep groups
        // b (< 8) in the first write and b + 8 in the second, lanes j >= 2 the
        // reverse; the low half of the wave writes step t, the high half t + 1.
        const int gA = 16 * (wave & 1) + ((lane >> 2) & 7), gB = gA + 8;
        const bool lowj = lj < 2;
        const int g1 = lowj ? gA : gB, g2 = lowj ? gB : gA;
#pragma unroll
        for (int t = 0; t < 16; t += 2) {
          uint2 o[2];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const half4_t bv = __builtin_bit_cast(half4_t, codeword_f16(kst[t + u], fp8));
            float4_t c = {0.f, 0.f, 0.f, 0.f};
            c = __builtin_amdgcn_mfma_f32_4x4x4f16(a_hi, bv, c, 0, 0, 0);
            c = __builtin_amdgcn_mfma_f32_4x4x4f16(a_lo, bv, c, 0, 0, 0);
            half4_t h;
            h[0] = static_cast<_Float16>(c[0]);
            h[1] = static_cast<_Float16>(c[1]);
            h[2] = static_cast<_Float16>(c[2]);
            h[3] = static_cast<_Float16>(c[3]);
            o[u] = __builtin_bit_cast(uint2, h);
          }
          // x: group gA of this lane's step, y: group gB of it
          const auto sx = __builtin_amdgcn_permlane32_swap(o[0].x, o[1].x, false, false);
          const auto sy = __builtin_amdgcn_permlane32_swap(o[0].y, o[1].y, false, false);
          const unsigned ax = sx[0], bx = sx[1], ay = sy[0], by = sy[1];
          const uint2 wa = make_uint2(ax, ay), wb = make_uint2(bx, by);
          const int code = cbase + 4 * ((t + (lane >> 5) + rot) & 15) + lj;
          *reinterpret_cast<uint2 *>(smem + code * 256 + g1 * 8) = lowj ? wa : wb;
          *reinterpret_cast<uint2 *>(smem + code * 256 + g2 * 8) = lowj ? wb : wa;
        }
      }
    };
    int *tctr = reinterpret_cast<int *>(smem + kTableCtr);
    if constexpr (APPEND) {
      // In the fused step the encoder team (waves 8..11) and the table waves
      // (0..7) run apart from here: the table waves meet through an LDS
      // counter, not workgroup barriers, so the team's encode never holds up
      // the tables, and the team waits for the tables only where it reads
      // them.  Its fp64 arithmetic then takes SIMD time in the setup, where
      // the SIMDs mostly wait for the parameter loads, instead of in the
      // token loop.  Values live on one path only (the team's loads, or the
      // rows of t_k_inv_t and the key codewords).  The band step's encode
      // reads no table (the new token's logit comes from the band), and its
      // scratch lies past the q' partial sums.
      if (wave >= 8) {
        if (sh < G) sink_logits();
        if (n_eff > 0) {
          const int p = S - 1;
          const size_t tokoff = subtile_offset(a, b, kv, p & ~15, bs_shift) + static_cast<size_t>(p & 15) * kL;
          if constexpr (BSTEP) {
            int phase = 0;  // shared by every copy of the meeting
            auto meet = [&] { team_sync(smem, ++phase); };
            step::encode_token<kD, KS, SQ, TBF>(a, *reinterpret_cast<step::Scratch<kD> *>(smem + kAppendScratch),
                                                b, kv, split, n_eff, tokoff, tid - 512, FP8, meet);
          } else {
            encode_items<TBF>(a, smem, b, kv, split, n_eff, tokoff, tid - 512, FP8, tctr);
          }
        }
        // the token loop reads the tables
        while (__hip_atomic_load(tctr, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < 16)
          __builtin_amdgcn_s_sleep(1);
      } else {
        q_partials();
        table_meet(tctr, 1);  // q' partial sums written
        build_tables();
        table_meet(tctr, 2);  // tables built
      }
    } else {
      // (The plain decode keeps workgroup barriers: with the waves apart, its
      // paged-cache decode at 32 x 32K tokens ran 26% slower.)
      if (sh >= 0 && sh < G) sink_logits();
      if (tid < 512) q_partials();
      __syncthreads();
      if (lut_wave) build_tables();
      __syncthreads();
    }
  }

  // Selector of the key-side MFMA: row block r of the accumulator receives the
  // table partials of sub-tile r (A[m][k] = 1 where m = 4r + k-row).
  half8_t asel[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const _Float16 one = ((lane & 15) == 4 * r + beta) ? static_cast<_Float16>(1.f) : static_cast<_Float16>(0.f);
    asel[r] = half8_t{one, one, one, one, one, one, one, one};
  }

  auto process_round = [&](const int R, const uint2 *kw, const uint2 *vw, const uint32_t ks, const uint32_t vq) {
    // K: partial logits gathered from the table by transposing reads; each
    // read hands lane (beta,u,v) four partials of (token R+16r+4beta+u, head v)
    // and serves as the B operand of a 16x16x32 MFMA (two steps per MFMA)
    // whose selector A sums them into accumulator row 4r+beta, column (u,v).
    // Lane (tau,u,v) then holds in register i the logit of token
    // R + 16 tau + 4 i + u for head v (log2 units), tau = lane >> 4.
    uint32_t w0[4], w1[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      w0[r] = __builtin_amdgcn_perm(kw[r].y, kw[r].x, rsel0);
      w1[r] = __builtin_amdgcn_perm(kw[r].y, kw[r].x, rsel1);
    }
    float4_t kacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int tp = 0; tp < 4; ++tp) {
      half8_t e[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t w = tp < 2 ? w0[r] : w1[r];
        const uint32_t kc = tp < 2 ? kc0 : kc1;
        const uint32_t ta = (2 * tp) & 3, tb = (2 * tp + 1) & 3;
        const half4_t lo = tr16_read(sbase + __builtin_amdgcn_perm(w, kc, 0x0C0C0000u | ((4u + ta) << 8) | ta));
        const half4_t hi = tr16_read(sbase + __builtin_amdgcn_perm(w, kc, 0x0C0C0000u | ((4u + tb) << 8) | tb));
        e[r] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) kacc = __builtin_amdgcn_mfma_f32_16x16x32_f16(asel[r], e[r], kacc, 0, 0, 0);
    }
    float z[4] = {kacc[0], kacc[1], kacc[2], kacc[3]};
    if constexpr (KS) {
      // the read path's per-token multiply: token R + 16 beta + 4 i + u's
      // scale is held by lane 16 beta + 4 i + u
#pragma unroll
      for (int i = 0; i < 4; ++i) z[i] *= __uint_as_float(static_cast<uint32_t>(__shfl(static_cast<int>(ks), 16 * beta + 4 * i + u)) << 16);
    }
    // scalar value arm: (scale, offset) of token R + 16 beta + 4 i + u
    float vsc[4] = {0.f, 0.f, 0.f, 0.f}, vzr[4] = {0.f, 0.f, 0.f, 0.f};
    if constexpr (SQ) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t w = static_cast<uint32_t>(__shfl(static_cast<int>(vq), 16 * beta + 4 * i + u));
        vsc[i] = __uint_as_float(w << 16) * 0x1p-8f;  // the value MFMA's B operand stays below 2^8 * scale
        vzr[i] = __uint_as_float(w & 0xffff0000u);
      }
    }
    if (R < t0 || R + 64 > t1) {  // ragged first or last round of the split
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tok = R + 16 * beta + 4 * i + u;
        if (tok < t0 || tok >= t1) {
          z[i] = -INFINITY;
          vsc[i] = vzr[i] = 0.f;  // rows past the tokens may hold anything
        }
      }
    }

    // online softmax over the round.  Accumulator column (u, v) of the value
    // MFMA mixes the four rows beta, so its reference max is shared by lanes
    // (beta, u, v), beta = 0..3; the four columns u of a head keep their own
    // maxima until the end of the unit.
    float zmax = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
    zmax = max_rows16(zmax);
    zmax = max_rows32(zmax);
    // The reference of a column moves only when its max exceeds it by more
    // than kLazyLog2, so the accumulator is rescaled rarely; probabilities
    // relative to a lagging reference stay below 2^kLazyLog2.  A column with
    // no attended token yet keeps reference -inf (exponent base taken as 0).
    const float m_new = fmaxf(m_run, zmax);
    const bool bump = m_new > m_run + kLazyLog2;
    const float ref = bump ? m_new : m_run;
    const float alpha = bump ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.f;
    const float base = ref == -INFINITY ? 0.f : ref;
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = __builtin_amdgcn_exp2f(z[i] - base);
    l_run = l_run * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
    if constexpr (SQ) z_run = z_run * alpha + ((p[0] * vzr[0] + p[1] * vzr[1]) + (p[2] * vzr[2] + p[3] * vzr[3]));
    if (__any(bump && m_run != -INFINITY)) {  // accumulators of -inf columns are zero
#pragma unroll
      for (int X = 0; X < 8; ++X) acc[X] *= alpha;
    }
    m_run = ref;
    half4_t pb;
    if constexpr (SQ) {
      pb = half4_t{static_cast<_Float16>(p[0] * vsc[0]), static_cast<_Float16>(p[1] * vsc[1]),
                   static_cast<_Float16>(p[2] * vsc[2]), static_cast<_Float16>(p[3] * vsc[3])};
    } else {
      pb = half4_t{static_cast<_Float16>(p[0]), static_cast<_Float16>(p[1]), static_cast<_Float16>(p[2]),
                   static_cast<_Float16>(p[3])};
    }
    const half4_t zero4 = {0, 0, 0, 0};

    // V: token sets s (tokens R + 16 beta + 4 i + s) in pairs; the A operand of
    // tile X holds coordinates of groups 8*(0..3) + X for the pair's 8 tokens
    // of each lane row, the B operand the matching probabilities of column
    // (set, head) = (u, v), zero where u is not the set.
#pragma unroll
    for (int sp = 0; sp < 2; ++sp) {
      const int s0 = 2 * sp, s1 = 2 * sp + 1;
      const half8_t bpair = __builtin_shufflevector(u == s0 ? pb : zero4, u == s1 ? pb : zero4, 0, 1, 2, 3, 4, 5, 6, 7);
      half8_t av[8];
#pragma unroll
      for (int X = 0; X < 8; ++X) {
        const uint32_t wa = X < 4 ? vw[s0].x : vw[s0].y;
        const uint32_t wb = X < 4 ? vw[s1].x : vw[s1].y;
        const uint32_t ca = (wa >> (8 * (X & 3))) & 0xffu;
        const uint32_t cb = (wb >> (8 * (X & 3))) & 0xffu;
        const half4_t lo = tr16_read(vbase + (ca << 5) + X * 8192);
        const half4_t hi = tr16_read(vbase + (cb << 5) + X * 8192);
        av[X] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
#pragma unroll
      for (int X = 0; X < 8; ++X) acc[X] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av[X], bpair, acc[X], 0, 0, 0);
    }
  };

  auto claim = [&]() -> int {
    int v = 0;
    if (lane == 0) v = __hip_atomic_fetch_add(rctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    return __builtin_amdgcn_readfirstlane(v);
  };
  int cur = wave;
  while (cur < nrounds) {
    const int nxt = claim();
    if (nxt < nrounds) load_round(R0 + 64 * nxt, kwb[1], vwb[1], ksb[1], vqb[1]);
    process_round(R0 + 64 * cur, kwb[0], vwb[0], ksb[0], vqb[0]);
    if (nxt >= nrounds) break;
    const int nxt2 = claim();
    if (nxt2 < nrounds) load_round(R0 + 64 * nxt2, kwb[0], vwb[0], ksb[0], vqb[0]);
    process_round(R0 + 64 * nxt, kwb[1], vwb[1], ksb[1], vqb[1]);
    cur = nxt2;
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
  float z_tot = 0.f;  // scalar value arm: the offsets' term of every coordinate of head v
  if constexpr (SQ) {
    z_tot = add_rows32(add_rows16(z_run)) * wcol;
    z_tot += row_ror<4>(z_tot);
    z_tot += row_ror<8>(z_tot);
  }
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

  // Rows of t_v for the combine are requested as soon as this wave's loop
  // ends, before the arrival is known: their latency hides behind the waves
  // still in the loop and the merge, and the last arrival finds them in
  // registers.
  load_tv_rows<TBF>(a, kv, tv);
  if constexpr (APPEND) {
    // the merge region holds the encoder team's scratch until its last item
    if (n_eff > 0 && wave < 8) {
      const int done = 4 * (BSTEP ? step::Tasks<kD, KS, SQ>::phases_of(split, n_eff) : team_phases(split, n_eff));
      int *ctr = reinterpret_cast<int *>(smem + kTeamCtr);
      while (__hip_atomic_load(ctr, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < done)
        __builtin_amdgcn_s_sleep(1);
    }
  }
  float *merge = reinterpret_cast<float *>(smem + kMergeBase);
  float *mw = merge + wave * kMergeFloats;
  if (lane < 4) {
    mw[lane] = m_run;
    mw[4 + lane] = l_tot;
  }
  if (u == 0) {
#pragma unroll
    for (int X = 0; X < 8; ++X)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        mw[8 + v * kMergeHead + kMergeBlk * beta + 4 * X + i] = SQ ? fmaf(acc[X][i], 256.f, z_tot) : acc[X][i];
  }
  __syncthreads();

  // ---- arrival (see the exchange below): counted now, while the waves merge
  const int bk = b * a.num_kv_heads + kv;
  if (a.n_split > 1 && tid == kCtl) {
    // the split's group (all splits when there is one group)
    int *ctl = reinterpret_cast<int *>(smem + kAuxCtl);
    const int gi = split / a.group_size;
    const int gsz = min(a.group_size, a.n_split - gi * a.group_size);
    int *cnt = a.counters + bk * (1 + a.n_group) + 1 + gi;
    const int last = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == gsz - 1;
    if (last) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    ctl[0] = last;
  }

  // ---- merge the waves into this split's partial (natural-log max), kept in
  // LDS and published to the exchange by the threads that form it
  float *own = reinterpret_cast<float *>(smem + kAuxOwn);
  float *ownml = reinterpret_cast<float *>(smem + kAuxCtl) + 8;
  const bool pub = a.n_split > 1 && act;
  uint64_t *slot = a.xch + (static_cast<size_t>(bk) * a.n_split + split) * kXchSlotWords;
  for (int i = tid; i < G * kD; i += WAVES * 64) {
    const int h = i / kD, d = i % kD;
    // all of this thread's reads first, then the arithmetic
    float mv[WAVES], lv[WAVES], av[WAVES];
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
      mv[w] = merge[w * kMergeFloats + h];
      lv[w] = merge[w * kMergeFloats + 4 + h];
      av[w] = merge[w * kMergeFloats + 8 + h * kMergeHead + (d >> 5) * kMergeBlk + (d & 31)];
    }
    float big = -INFINITY;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) big = fmaxf(big, mv[w]);
    float num = 0.f, den = 0.f;
    if (big != -INFINITY) {
#pragma unroll
      for (int w = 0; w < WAVES; ++w) {
        const float wt = (mv[w] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mv[w] - big);
        num = fmaf(wt, av[w], num);
        den = fmaf(wt, lv[w], den);
      }
    }
    // kept and published as (log-sum-exp, 1, normalised partial), so that the
    // combining split takes its own partial with the bits the others read
    const float lse = den > 0.f ? big * kLn2 + __logf(den) : -INFINITY;
    const float o = den > 0.f ? num / den : 0.f;
    own[i] = o;
    if (d == 0) {
      ownml[2 * h] = lse;
      ownml[2 * h + 1] = 1.f;
    }
    if (pub) {
      put_word(a.epoch, slot + 2 * G + i, o);
      if (d == 0) put_word(a.epoch, slot + 2 * h, lse);
    }
  }
}

// The combining split of a (sequence, KV head): log-sum-exp merge of the
// splits' partials, the sink added once with its shift -(q . k_bar) * scale
// (Lemma S1; appendix on attention sinks), the new token of a fused step,
// division by the denominator, and the inverse value transform
// out = s_hat t_v^T (Corollary 1).  The split's own partial and blocks of the
// new token are read from LDS, the other splits' from the exchange (every
// word's tag checked against the call's epoch); splits that attend to no
// token published no partial and are skipped.
// Rows of the band attended by split `split` of n_split: consecutive shares
// in split order.
__device__ __forceinline__ void band_share(const int nband, const int n_split, const int split, int &first,
                                           int &count) {
  const int per = (nband + n_split - 1) / n_split;
  first = min(nband, split * per);
  count = min(nband, first + per) - first;
}

// Exchange slots whose words one combine requests before it waits.  The
// combine runs once per (sequence, KV head) from a cold instruction cache, so
// its code is kept short: four slots per batch, and many splits are merged in
// groups (two levels) rather than read in long batches by one workgroup.
#ifndef NOVA_KV_XCH_BATCH
#define NOVA_KV_XCH_BATCH 4
#endif
constexpr int kXchBatch = NOVA_KV_XCH_BATCH;
static_assert(kXchBatch <= 48, "a batch's requests stay within the wave's outstanding-load count");

__device__ __forceinline__ uint64_t readlane64(const uint64_t x, const int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(x)), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(x >> 32)), lane);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Reads `count` (1..kXchBatch) exchange slots and hands each wanted one, in
// batch order, to take(i, log-sum-exp, normalised partial) for head h,
// coordinate `tid` (h = tid / 128).  The heads' log-sum-exp words are
// requested one slot per lane and broadcast from that lane; each thread
// requests its coordinate of every slot.  All requests are issued before the
// first wait, so the batch costs one round trip; past `count` they repeat the
// last slot.  If a word of the wave's batch does not carry the call's tag
// yet, the wave reads the batch again slot by slot, waiting for each word.
// Returns false if a word never arrived (not expected).
template <class SlotOf, class Want, class Take>
__device__ __forceinline__ bool read_slots(const uint32_t epoch, const int count, const int h, const int G,
                                           const int tid, SlotOf slot_of, Want want, Take take) {
  if (count <= 0) return true;
  const int lane = tid & 63;
  const uint64_t lw = get_word(slot_of(min(lane, count - 1)) + 2 * h);
  uint64_t wa[kXchBatch];
#pragma unroll
  for (int i = 0; i < kXchBatch; ++i) wa[i] = get_word(slot_of(min(i, count - 1)) + 2 * G + tid);
  bool ready = lane >= count || !want(lane) || word_ready(epoch, lw);
#pragma unroll
  for (int i = 0; i < kXchBatch; ++i)
    if (i < count && want(i) && !word_ready(epoch, wa[i])) ready = false;
  if (__all(ready)) {
#pragma unroll
    for (int i = 0; i < kXchBatch; ++i)
      if (i < count && want(i)) take(i, word_value(readlane64(lw, i)), word_value(wa[i]));
    return true;
  }
  bool ok = true;
  for (int i = 0; i < count; ++i) {
    if (!want(i)) continue;
    const uint64_t *sp = slot_of(i);
    uint64_t wm = get_word(sp + 2 * h), w = get_word(sp + 2 * G + tid);
    for (int n = 0; !(word_ready(epoch, wm) && word_ready(epoch, w)); ++n) {
      if (n == kSpinLimit) {
        ok = false;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
      wm = get_word(sp + 2 * h);
      w = get_word(sp + 2 * G + tid);
    }
    take(i, word_value(wm), word_value(w));
  }
  return ok;
}

// The partials this combine reads: the unit's split slots (one level), or
// the slots of its split groups (two levels).
struct Slots {
  uint64_t *base;        // slot 0
  int n, own;            // number of slots, this workgroup's slot
  bool all_valid;        // group slots: every slot holds a partial and a band block
};

// Empties n slots from base on (heads 0..G-1; the band blocks too when the
// call has a band).  Called once every read of the slots in this workgroup
// is done (after a barrier); the words of the other workgroups were read, so
// their stores precede these.
__device__ __forceinline__ void clear_slots(uint64_t *base, const int n, const int G, const int tid,
                                            const bool band) {
  if (tid >= G * kD) return;
  for (int j = 0; j < n; ++j) {
    uint64_t *sp = base + static_cast<size_t>(j) * kXchSlotWords;
    clear_word(sp + 2 * G + tid);
    if (tid < 2 * G) clear_word(sp + tid);
    if (band) {
      clear_word(sp + kXchBandWords + 2 * G + tid);
      if (tid < 2 * G) clear_word(sp + kXchBandWords + tid);
    }
  }
}

template <int WAVES, bool APPEND, bool BSTEP, bool TBF>
__device__ __forceinline__ void combine_unit(const DecodeArgs &a, uint8_t *smem, const int b, const int kv,
                                             const int bk, const size_t row0, const int own_split, const int S,
                                             const int lo, const int tend, const int n_eff, const int band_lo,
                                             const int sink_end, const T4 (&tv)[8], const Slots sl) {
  const int tid = threadIdx.x;
  const int G = a.gqa;
  // Sink-plus-recent band: positions [band_lo, sink_end) and [tend, S) (the
  // splits read [lo, tend) from the pools).  Every split attended its share
  // of the band rows (its partial is in LDS for this split, in the exchange
  // for the others); the shares are merged in split order and taken after
  // the splits as one more partial, whose value term is in the original
  // domain.
  using BL = BandLds<kD, 4, WAVES>;
  const int nband = a.band_k ? max(0, sink_end - band_lo) + (S - tend) : 0;
  float *bout = reinterpret_cast<float *>(smem + BL::kPart);  // [4][128] band term of the output
  float *shat = reinterpret_cast<float *>(smem + kAuxQ);    // [4][128]
  float *outp = reinterpret_cast<float *>(smem + kAuxOut);  // [part][head][128]
  float *ctlf = reinterpret_cast<float *>(smem + kAuxCtl);
  const float *own = reinterpret_cast<const float *>(smem + kAuxOwn);
  const int d = tid & (kD - 1), jp = tid >> 7;  // tv holds row d of t_v, columns 32*jp .. 32*jp+31
  if (tid < G * kD) {
    const int h = tid >> 7;
    const float sk = ctlf[4 + h];
    bool ok = true;
    // fused step: the new token's block results, requested with the splits'
    // partials (blocks of this split from LDS)
    float zp[4] = {0.f, 0.f, 0.f, 0.f}, vp = 0.f;
    const float *res = reinterpret_cast<const float *>(smem + kItemRes);
    uint64_t *xn = a.xnew + static_cast<size_t>(bk) * 8 * 32;
    const int vj = (4 + (d >> 5)) * 32 + (d & 31);
    uint64_t wz[4], wv;
    constexpr bool new_term = APPEND && !BSTEP;  // with a band the new token is a band row
    if constexpr (new_term) {
#pragma unroll
      for (int k = 0; k < 4; ++k) wz[k] = get_word(xn + k * 32 + h);
      wv = get_word(xn + vj);
    }
    // online log-sum-exp over the splits, the sink counted once
    float big = sk, num = 0.f, den = sk == -INFINITY ? 0.f : 1.f;
    auto take = [&](float ms, float ls, float as) {
      if (ms == -INFINITY) return;
      if (ms > big) {
        const float f = big == -INFINITY ? 0.f : __expf(big - ms);
        num *= f;
        den *= f;
        big = ms;
      }
      const float w = __expf(ms - big);
      den = fmaf(w, ls, den);
      num = fmaf(w, as, num);
    };
    // splits (or groups) in index order whichever split combines, so the
    // result does not depend on the arrival order; the other slots are read
    // kXchBatch at a time
    uint64_t *xs = sl.base;
    const int n_oth = sl.n - 1;
    const int own_slot = sl.own;
    bool own_done = false;
    auto take_own = [&]() {
      take(ctlf[8 + 2 * h], ctlf[8 + 2 * h + 1], own[tid]);
      own_done = true;
    };
    for (int k0 = 0; k0 < n_oth; k0 += kXchBatch) {
      auto sidx = [&](int i) { return k0 + i + (k0 + i >= own_slot ? 1 : 0); };
      ok &= read_slots(
          a.epoch, min(kXchBatch, n_oth - k0), h, G, tid,
          [&](int i) { return xs + static_cast<size_t>(sidx(i)) * kXchSlotWords; },
          [&](int i) { return sl.all_valid || lo + sidx(i) * a.chunk < tend; },
          [&](int i, float ms, float as) {
            if (!own_done && sidx(i) > own_slot) take_own();
            take(ms, 1.f, as);
          });
    }
    if (!own_done) take_own();
    if constexpr (new_term) {
      if (S > 0) {  // the new token, after the splits
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (k % n_eff == own_split) {
            zp[k] = res[k * 32 + h];
          } else {
            for (int n = 0; !word_ready(a.epoch, wz[k]); ++n) {
              if (n == kSpinLimit) {
                ok = false;
                break;
              }
              __builtin_amdgcn_s_sleep(2);
              wz[k] = get_word(xn + k * 32 + h);
            }
            zp[k] = word_value(wz[k]);
          }
        }
        if ((4 + (d >> 5)) % n_eff == own_split) {
          vp = res[vj];
        } else {
          for (int n = 0; !word_ready(a.epoch, wv); ++n) {
            if (n == kSpinLimit) {
              ok = false;
              break;
            }
            __builtin_amdgcn_s_sleep(2);
            wv = get_word(xn + vj);
          }
          vp = word_value(wv);
        }
        take((((zp[0] + zp[1]) + zp[2]) + zp[3]) * kLn2, 1.f, vp);
      }
    }
    float bo = 0.f;
    if (nband > 0) {  // the band, after the splits (and the new token)
      // the splits' (or groups') shares in index order, this split's from LDS
      float mb = -INFINITY, lb = 0.f, ab = 0.f;
      auto take_b = [&](float ms, float ls, float as) {
        if (ms == -INFINITY) return;  // a group without band rows
        if (ms > mb) {
          const float f = mb == -INFINITY ? 0.f : __expf(mb - ms);
          lb *= f;
          ab *= f;
          mb = ms;
        }
        const float w = __expf(ms - mb);
        lb = fmaf(w, ls, lb);
        ab = fmaf(w, as, ab);
      };
      auto has_share = [&](int sp) {
        if (sl.all_valid) return true;
        int first, count;
        band_share(nband, a.n_split, sp, first, count);
        return count > 0;
      };
      const float *bst = reinterpret_cast<const float *>(smem + BL::kStat);
      const float *bzs = reinterpret_cast<const float *>(smem + BL::kZ);
      bool own_b = false;
      auto take_own_b = [&]() {
        if (has_share(own_slot)) take_b(bst[h], bst[4 + h], bzs[h * kD + d]);
        own_b = true;
      };
      for (int k0 = 0; k0 < n_oth; k0 += kXchBatch) {
        auto sidx = [&](int i) { return k0 + i + (k0 + i >= own_slot ? 1 : 0); };
        ok &= read_slots(
            a.epoch, min(kXchBatch, n_oth - k0), h, G, tid,
            [&](int i) { return xs + static_cast<size_t>(sidx(i)) * kXchSlotWords + kXchBandWords; },
            [&](int i) { return has_share(sidx(i)); },
            [&](int i, float ms, float as) {
              if (!own_b && sidx(i) > own_slot) take_own_b();
              take_b(ms, 1.f, as);
            });
      }
      if (!own_b) take_own_b();
      if (mb > big) {
        const float f = big == -INFINITY ? 0.f : __expf(big - mb);
        num *= f;
        den *= f;
        big = mb;
      }
      const float wb = mb == -INFINITY ? 0.f : __expf(mb - big);
      den = fmaf(wb, lb, den);
      bo = wb * ab;
    }
    // a word that never arrived (not expected) leaves this row NaN
    shat[tid] = !ok ? __builtin_nanf("") : (den > 0.f ? num / den : 0.f);
    bout[tid] = den > 0.f ? bo / den : 0.f;
  } else if (tid < 4 * kD) {
    shat[tid] = 0.f;
  }
  __syncthreads();
  if (a.clear_xch && a.n_split > 1) {  // captured call: empty the unit's exchange words, all read
    clear_slots(sl.base, sl.n, G, tid, nband > 0);
    if (APPEND && tid < 8 * 32) clear_word(a.xnew + static_cast<size_t>(bk) * 8 * 32 + tid);
  }
  if (tid < 512) {
    // all eight values of a head are requested before they are used
    float o[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      float4 sv[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) sv[i] = *reinterpret_cast<const float4 *>(shat + h * kD + 32 * jp + 4 * i);
      float x = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float4 t = t4_value(tv[i], TBF);
        x = fmaf(sv[i].x, t.x, x);
        x = fmaf(sv[i].y, t.y, x);
        x = fmaf(sv[i].z, t.z, x);
        x = fmaf(sv[i].w, t.w, x);
      }
      o[h] = x;
    }
#pragma unroll
    for (int h = 0; h < 4; ++h) outp[(jp * 4 + h) * kD + d] = o[h];
  }
  __syncthreads();
  if (tid < G * kD) {
    const int h = tid >> 7;
    const float o =
        (outp[h * kD + d] + outp[(4 + h) * kD + d]) + (outp[(8 + h) * kD + d] + outp[(12 + h) * kD + d]);
    a.out[(row0 + h) * kD + d] = nband > 0 ? o + bout[tid] : o;
  }
}

// Two-level combine (many splits): the last split of each group of
// a.group_size splits merges its group's partials, in split order, into one
// partial (its code part and its band part), keeps it in LDS in place of its
// own and publishes it to the group's slot; the last group then combines the
// group slots.  No sink, new token or inverse transform at this level.
template <int WAVES>
__device__ __forceinline__ void merge_group(const DecodeArgs &a, uint8_t *smem, const int bk, const int split,
                                            const int S, const int lo, const int tend, const int band_lo,
                                            const int sink_end) {
  const int tid = threadIdx.x;
  const int G = a.gqa;
  using BL = BandLds<kD, 4, WAVES>;
  const int nband = a.band_k ? max(0, sink_end - band_lo) + (S - tend) : 0;
  const int gi = split / a.group_size;
  const int g0 = gi * a.group_size, gsz = min(a.group_size, a.n_split - g0);
  float *ctlf = reinterpret_cast<float *>(smem + kAuxCtl);
  float *own = reinterpret_cast<float *>(smem + kAuxOwn);
  float *bst = reinterpret_cast<float *>(smem + BL::kStat);
  float *bz = reinterpret_cast<float *>(smem + BL::kZ);
  uint64_t *xs = a.xch + static_cast<size_t>(bk) * a.n_split * kXchSlotWords;
  uint64_t *gslot = a.xgrp + (static_cast<size_t>(bk) * a.n_group + gi) * kXchSlotWords;
  const bool mine = tid < G * kD;
  const int h = tid >> 7, d = tid & (kD - 1);
  float big = -INFINITY, den = 0.f, num = 0.f;  // the group's code partial
  float mb = -INFINITY, lb = 0.f, ab = 0.f;     // the group's band partial
  if (mine) {
    bool ok = true;
    auto lse = [](float &m, float &l, float &acc, const float ms, const float ls, const float as) {
      if (ms == -INFINITY) return;
      if (ms > m) {
        const float f = m == -INFINITY ? 0.f : __expf(m - ms);
        acc *= f;
        l *= f;
        m = ms;
      }
      const float w = __expf(ms - m);
      l = fmaf(w, ls, l);
      acc = fmaf(w, as, acc);
    };
    // the group's other splits in split order, this split's partial from LDS
    const int own_i = split - g0;
    auto sidx = [&](int i) { return g0 + i + (i >= own_i ? 1 : 0); };
    bool own_done = false, own_b = false;
    for (int k0 = 0; k0 < gsz - 1; k0 += kXchBatch)
      ok &= read_slots(
          a.epoch, min(kXchBatch, gsz - 1 - k0), h, G, tid,
          [&](int i) { return xs + static_cast<size_t>(sidx(k0 + i)) * kXchSlotWords; },
          [&](int i) { return lo + sidx(k0 + i) * a.chunk < tend; },
          [&](int i, float ms, float as) {
            if (!own_done && k0 + i >= own_i) {
              lse(big, den, num, ctlf[8 + 2 * h], ctlf[8 + 2 * h + 1], own[tid]);
              own_done = true;
            }
            lse(big, den, num, ms, 1.f, as);
          });
    if (!own_done) lse(big, den, num, ctlf[8 + 2 * h], ctlf[8 + 2 * h + 1], own[tid]);
    // band shares of the group's splits, in split order
    if (nband > 0) {
      auto has_share = [&](int sp) {
        int first, count;
        band_share(nband, a.n_split, sp, first, count);
        return count > 0;
      };
      auto take_own_b = [&]() {
        if (has_share(split)) lse(mb, lb, ab, bst[h], bst[4 + h], bz[h * kD + d]);
        own_b = true;
      };
      for (int k0 = 0; k0 < gsz - 1; k0 += kXchBatch)
        ok &= read_slots(
            a.epoch, min(kXchBatch, gsz - 1 - k0), h, G, tid,
            [&](int i) { return xs + static_cast<size_t>(sidx(k0 + i)) * kXchSlotWords + kXchBandWords; },
            [&](int i) { return has_share(sidx(k0 + i)); },
            [&](int i, float ms, float as) {
              if (!own_b && k0 + i >= own_i) take_own_b();
              lse(mb, lb, ab, ms, 1.f, as);
            });
      if (!own_b) take_own_b();
    }
    if (!ok) num = __builtin_nanf("");  // a word that never arrived (not expected): the rows turn NaN
    // published (and kept) in the splits' form: (log-sum-exp, 1, normalised partial)
    num = den > 0.f ? num / den : num;
    big = den > 0.f ? big + __logf(den) : -INFINITY;
    den = 1.f;
    ab = lb > 0.f ? ab / lb : 0.f;
    mb = lb > 0.f ? mb + __logf(lb) : -INFINITY;
    lb = 1.f;
    put_word(a.epoch, gslot + 2 * G + tid, num);
    if (d == 0) put_word(a.epoch, gslot + 2 * h, big);
    if (nband > 0) {
      put_word(a.epoch, gslot + kXchBandWords + 2 * G + tid, ab);
      if (d == 0) put_word(a.epoch, gslot + kXchBandWords + 2 * h, mb);
    }
  }
  __syncthreads();  // every read of this split's own partial and of the group's slots is done
  if (a.clear_xch) clear_slots(xs + static_cast<size_t>(g0) * kXchSlotWords, gsz, G, tid, nband > 0);
  // the group's partial replaces this split's own
  if (mine) {
    own[tid] = num;
    bz[h * kD + d] = ab;
    if (d == 0) {
      ctlf[8 + 2 * h] = big;
      ctlf[8 + 2 * h + 1] = den;
      bst[h] = mb;
      bst[4 + h] = lb;
    }
  }
}

// One workgroup per (sequence, KV head, split).  Every split publishes its
// partial to the exchange and counts its arrival; the last one combines.
// The arrival counters live in the workspace and the last split resets its
// counter to 0, so a decode step is a single launch.
// TBF: the transforms are stored as bf16 (NOVA_KV_BF16_TRANSFORMS).
template <int WAVES, bool APPEND, bool KS, bool FP8, bool SQ, bool BSTEP, bool TBF>
__global__ void __launch_bounds__(WAVES * 64) decode_lut_d128(DecodeArgs a) {
  static_assert(!BSTEP || APPEND, "a band step is a fused step");
  static_assert(!APPEND || BSTEP || !(KS || SQ), "without a band the fused step serves the plain and fp8 formats");
  static_assert(WAVES == 12, "the exchange roles assume 12 waves");
  __shared__ __attribute__((aligned(16))) uint8_t smem[lds_bytes<WAVES, APPEND>()];
  const int tid = threadIdx.x;
  // each XCD takes a contiguous range of the logical workgroup order
  int kv, b, split;
  unit_of_workgroup(xcd_contiguous(blockIdx.x, gridDim.x), a.n_split, a.b_chunk, a.num_kv_heads, kv, b, split);
  const int rest = b * a.n_split + split;  // distinct among the workgroups of a KV head
  const int bk = b * a.num_kv_heads + kv;
  const int G = a.gqa;

  const int S = a.seq_lens[b];
  const int att_lo = a.window > 0 ? max(0, S - a.window) : 0;
  // The pools are read for [lo, tend): the attended span without the band.
  // A fused step without a band attends its newest token from the step's own
  // codes, so the pools are read for [att_lo, S - 1); with a band that token
  // is the band's last row.
  const AttendedSpans spn = attended_spans(att_lo, S, a.n_sink, a.n_rec);
  constexpr bool new_from_codes = APPEND && !BSTEP;
  const int lo = new_from_codes ? att_lo : spn.code_lo;
  const int tend = new_from_codes ? max(S - 1, att_lo) : spn.code_hi;
  const int t0 = lo + split * a.chunk;  // splits tile the span read from the pools
  const int t1 = min(tend, lo + (split + 1) * a.chunk);
  const size_t row0 = static_cast<size_t>(b) * a.num_q_heads + kv * G;
  // Fused step: the splits with pool tokens (at least split 0) share the encode
  // of the new token; such a split runs the setup even with no token of its own.
  int n_eff = 1;
  bool items = false;
  if (APPEND && S > 0) {
    const int n_act = tend > lo ? (tend - lo + a.chunk - 1) / a.chunk : 0;
    n_eff = max(n_act, 1);
    items = split < n_eff;
  }

  T4 tv[8];
  split_pass<WAVES, APPEND, KS, FP8, SQ, BSTEP, TBF>(a, smem, b, kv, split, t0, max(t0, t1), row0, rest, items ? n_eff : 0, S, tv);
  // Sink-plus-recent band: this split's share of the band rows, attended in
  // the table's LDS region (free after the split pass) and published beside
  // the split's partial; one CU would read the whole band at a fraction of
  // the HBM rate, so the shares spread it over the unit's workgroups.
  const int nband = a.band_k ? max(0, spn.sink_end - att_lo) + (S - tend) : 0;
  int bfirst = 0, bcount = 0;
  if (nband > 0) {
    band_share(nband, a.n_split, split, bfirst, bcount);
    if (bcount > 0) {
      using BL = BandLds<kD, 4, WAVES>;
      if constexpr (BSTEP) {
        // a fused step's new token is the band's last row: the split that
        // attends it stores it, and reads it back after the barrier
        if (bfirst + bcount == nband) {
          step::store_band_rows<kD>(a, b, kv, S - 1);
          __syncthreads();
        }
      }
      band_attention<kD, 4, WAVES, WAVES>(a, smem, b, kv, row0, att_lo, spn.sink_end, tend, S, bfirst, bcount,
                                          reinterpret_cast<const float *>(smem + kAuxQ),
                                          reinterpret_cast<const float *>(smem + kItemRes));
      // the share is kept and published as (log-sum-exp, 1, normalised partial)
      float *bst = reinterpret_cast<float *>(smem + BL::kStat);
      float *bz = reinterpret_cast<float *>(smem + BL::kZ);
      const int h = tid >> 7;
      float lse = 0.f, o = 0.f;
      if (tid < G * kD) {
        const float lb = bst[4 + h];
        lse = lb > 0.f ? bst[h] + __logf(lb) : -INFINITY;
        o = lb > 0.f ? bz[tid] / lb : 0.f;
      }
      __syncthreads();
      if (tid < G * kD) {
        bz[tid] = o;
        if ((tid & (kD - 1)) == 0) {
          bst[h] = lse;
          bst[4 + h] = 1.f;
        }
        if (a.n_split > 1) {
          uint64_t *bw = a.xch + (static_cast<size_t>(bk) * a.n_split + split) * kXchSlotWords + kXchBandWords;
          put_word(a.epoch, bw + 2 * G + tid, o);
          if ((tid & (kD - 1)) == 0) put_word(a.epoch, bw + 2 * h, lse);
        }
      }
    }
  }
  int *ctl = reinterpret_cast<int *>(smem + kAuxCtl);
  __syncthreads();  // the split's partial and its blocks of the new token are in LDS; the count is known
  if (a.n_split > 1) {
    if (ctl[0] == 0) return;
  }
  uint64_t *xs = a.xch + static_cast<size_t>(bk) * a.n_split * kXchSlotWords;
  if (a.n_group > 1) {
    // two levels: merge this split's group, then count the group in
    merge_group<WAVES>(a, smem, bk, split, S, lo, tend, att_lo, spn.sink_end);
    if (tid == kCtl) {
      int *cnt = a.counters + bk * (1 + a.n_group);
      const int last =
          __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == a.n_group - 1;
      if (last) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      ctl[0] = last;
    }
    __syncthreads();
    if (ctl[0] == 0) return;
    const Slots gs{a.xgrp + static_cast<size_t>(bk) * a.n_group * kXchSlotWords, a.n_group, split / a.group_size,
                   true};
    combine_unit<WAVES, APPEND, BSTEP, TBF>(a, smem, b, kv, bk, row0, split, S, lo, tend, n_eff, att_lo, spn.sink_end, tv, gs);
  } else {
    combine_unit<WAVES, APPEND, BSTEP, TBF>(a, smem, b, kv, bk, row0, split, S, lo, tend, n_eff, att_lo, spn.sink_end, tv,
                                Slots{xs, a.n_split, split, false});
  }
}

}  // namespace

bool lut_path_eligible(int head_dim, int gqa, int block_size) {
  return block_size % 16 == 0 && ((head_dim == 128 && gqa <= 4) || (head_dim == 64 && gqa <= 8));
}

// Splits per (sequence, KV head): enough for about 256 workgroups, one per
// CU, but never fewer than kMinChunk tokens per split.  Every split pays the
// whole setup (parameters, query transform, tables) and adds a partial to the
// combine, so a short span is not worth many CUs: a split of kMinChunk tokens
// streams its codes in less time than one more partial costs the combine.
#ifndef NOVA_KV_MIN_CHUNK
#define NOVA_KV_MIN_CHUNK 512
#endif
constexpr int kMinChunk = NOVA_KV_MIN_CHUNK;

void plan_lut(int batch, int num_kv_heads, int max_seq_len, int *n_split, int *chunk) {
  const long long units = static_cast<long long>(batch) * num_kv_heads;
  int ns = static_cast<int>((256 + units - 1) / units);
  if (ns < 1) ns = 1;
  int ch = (max_seq_len + ns - 1) / ns;
  ch = (ch + 63) & ~63;
  if (ch < kMinChunk) ch = kMinChunk;
  *chunk = ch;
  *n_split = (max_seq_len + ch - 1) / ch;
}

// Sequences per block of the table kernels' workgroup order: the largest
// divisor of batch that leaves about two KV heads (all their splits) in each
// XCD's eighth of the grid.  Same-box timing at B=8, 8 KV heads, 4 splits:
// two KV heads per XCD beat both one (32 CUs of one L2 request the same
// parameter lines at once) and eight (every L2 fetches every KV head's
// parameters).
// One combine reads up to kXchBatch other slots in one round trip; above
// that the splits are merged in groups of about sqrt(n_split) splits (a power
// of two, at most 32) first.
#ifndef NOVA_KV_ONE_LEVEL_MAX
#define NOVA_KV_ONE_LEVEL_MAX (kXchBatch + 1)
#endif
#ifndef NOVA_KV_GROUP_MAX
#define NOVA_KV_GROUP_MAX 32
#endif
int plan_group_size(int n_split) {
  if (n_split <= NOVA_KV_ONE_LEVEL_MAX) return n_split > 0 ? n_split : 1;
  int gs = 2;
  while (gs < NOVA_KV_GROUP_MAX && gs * gs < n_split) gs *= 2;
  return gs;
}

int plan_b_chunk(int batch, int num_kv_heads, int n_split) {
  const long long grid = static_cast<long long>(batch) * num_kv_heads * n_split;
  const long long per_xcd = grid / 8 > 0 ? grid / 8 : 1;
  long long target = per_xcd / (2LL * n_split);
  if (target < 1) target = 1;
  int bc = 1;
  for (int d = 1; d <= batch && d <= target; ++d)
    if (batch % d == 0) bc = d;
  return bc;
}

template <bool APPEND, bool KS, bool BSTEP, bool TBF>
void launch_d128(const DecodeArgs &a, const dim3 grid, const dim3 block, hipStream_t stream) {
  constexpr int W = 12;
  if (a.v_sq) {
    if (a.cb_fp8)
      decode_lut_d128<W, APPEND, KS, true, true, BSTEP, TBF><<<grid, block, 0, stream>>>(a);
    else
      decode_lut_d128<W, APPEND, KS, false, true, BSTEP, TBF><<<grid, block, 0, stream>>>(a);
  } else {
    if (a.cb_fp8)
      decode_lut_d128<W, APPEND, KS, true, false, BSTEP, TBF><<<grid, block, 0, stream>>>(a);
    else
      decode_lut_d128<W, APPEND, KS, false, false, BSTEP, TBF><<<grid, block, 0, stream>>>(a);
  }
}

template <bool TBF>
void launch_d128_storage(const DecodeArgs &a, const dim3 grid, const dim3 block, hipStream_t stream) {
  if (a.append && a.band_k)
    a.k_scales ? launch_d128<true, true, true, TBF>(a, grid, block, stream)
               : launch_d128<true, false, true, TBF>(a, grid, block, stream);
  else if (a.append)  // plain or fp8 codebooks (checked by the caller)
    a.cb_fp8 ? decode_lut_d128<12, true, false, true, false, false, TBF><<<grid, block, 0, stream>>>(a)
             : decode_lut_d128<12, true, false, false, false, false, TBF><<<grid, block, 0, stream>>>(a);
  else
    a.k_scales ? launch_d128<false, true, false, TBF>(a, grid, block, stream)
               : launch_d128<false, false, false, TBF>(a, grid, block, stream);
}

hipError_t launch_decode_lut(const DecodeArgs &a, hipStream_t stream) {
  // A fused step in the key-scale or scalar value format, or with a band,
  // attends its new token as the band's last row: it needs a recent band.
  if (a.append && (a.k_scales || a.v_sq || a.band_k) && !(a.band_k && a.n_rec >= 1)) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(a.batch * a.num_kv_heads * a.n_split));
  const dim3 block(12 * 64);
  a.t_bf16 ? launch_d128_storage<true>(a, grid, block, stream) : launch_d128_storage<false>(a, grid, block, stream);
  return hipGetLastError();
}

}  // namespace novakv
