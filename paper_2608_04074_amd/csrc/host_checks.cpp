// Host-side validation of the C ABI (plain C++: built into libnovakv and, by
// the tests, into a sanitizer-checked host program).
#include "host_checks.h"

#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <atomic>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

namespace novakv {
namespace host {

thread_local std::string g_last_error;

nova_kv_status fail(nova_kv_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

nova_kv_status ok() {
  g_last_error.clear();
  return NOVA_KV_OK;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Tag of the split exchange of the next decode call: every call gets a new
// nonzero number (the workspace's words of one call are never taken for
// another's; zero marks a never-written word).  A captured call's replays
// all carry its epoch and empty what they exchange; its epoch is even, so no
// directly launched call (odd epochs, whose words stay) ever shares it.
uint32_t next_epoch(bool captured) {
  static std::atomic<uint32_t> counter{0};
  uint32_t e;
  do {
    const uint32_t c = counter.fetch_add(1, std::memory_order_relaxed);
    e = captured ? (c + 1) << 1 : (c << 1) | 1u;
  } while (e == 0);
  return e;
}

nova_kv_status check_params(const nova_kv_params *p, bool need_encode, bool need_decode) {
  if (!p) return fail(NOVA_KV_ERR_INVALID_ARG, "params is NULL");
  if (p->num_kv_heads <= 0) return fail(NOVA_KV_ERR_INVALID_ARG, "num_kv_heads must be > 0");
  if (p->group_dim <= 0 || p->head_dim <= 0 || p->head_dim % p->group_dim != 0)
    return fail(NOVA_KV_ERR_INVALID_ARG, "head_dim (%d) must be a positive multiple of group_dim (%d)",
                p->head_dim, p->group_dim);
  if (p->codebook_size <= 0) return fail(NOVA_KV_ERR_INVALID_ARG, "codebook_size must be > 0");
  if (p->group_dim != novakv::kGroupDim)
    return fail(NOVA_KV_ERR_UNSUPPORTED, "group_dim %d unsupported (only 4)", p->group_dim);
  if (p->codebook_size != novakv::kCodebookSize)
    return fail(NOVA_KV_ERR_UNSUPPORTED, "codebook_size %d unsupported (only 256)", p->codebook_size);
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(NOVA_KV_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", p->head_dim);
  if ((p->flags & ~(NOVA_KV_KEY_SCALE | NOVA_KV_FP8_CODEBOOKS | NOVA_KV_SQ_VALUES | NOVA_KV_BF16_TRANSFORMS)) != 0)
    return fail(NOVA_KV_ERR_UNSUPPORTED,
                "flags 0x%x unsupported (NOVA_KV_KEY_SCALE, NOVA_KV_FP8_CODEBOOKS, NOVA_KV_SQ_VALUES, "
                "NOVA_KV_BF16_TRANSFORMS)", p->flags);
  const bool sq = (p->flags & NOVA_KV_SQ_VALUES) != 0;  // cb_v unused
  if (!p->kbar || !p->cb_k || (!sq && !p->cb_v)) return fail(NOVA_KV_ERR_INVALID_ARG, "kbar/cb_k/cb_v is NULL");
  if (!aligned(p->cb_k, 16) || (!sq && !aligned(p->cb_v, 16)))
    return fail(NOVA_KV_ERR_INVALID_ARG, "codebooks must be 16-byte aligned");
  if (need_encode && (!p->t_k || !p->t_v)) return fail(NOVA_KV_ERR_INVALID_ARG, "t_k/t_v is NULL");
  if (need_decode && (!p->t_k_inv_t || !p->t_v))
    return fail(NOVA_KV_ERR_INVALID_ARG, "t_k_inv_t/t_v is NULL");
  if (!aligned(p->kbar, 16) || !aligned(p->t_v, 16) || (need_encode && !aligned(p->t_k, 16)) ||
      (need_decode && !aligned(p->t_k_inv_t, 16)))
    return fail(NOVA_KV_ERR_INVALID_ARG, "kbar and transforms must be 16-byte aligned");
  return NOVA_KV_OK;
}

nova_kv_status check_layout(const nova_kv_layout *lay) {
  if (!lay) return fail(NOVA_KV_ERR_INVALID_ARG, "layout is NULL");
  if (lay->block_size <= 0 || lay->blocks_per_seq <= 0)
    return fail(NOVA_KV_ERR_INVALID_ARG, "block_size and blocks_per_seq must be > 0");
  if (static_cast<long long>(lay->block_size) * lay->blocks_per_seq > (1LL << 30))
    return fail(NOVA_KV_ERR_INVALID_ARG, "per-sequence capacity too large");
  return NOVA_KV_OK;
}

// The scale pool of the key-scale format (ignored otherwise).
nova_kv_status check_scales(const nova_kv_params *p, const void *k_scales) {
  if (!(p->flags & NOVA_KV_KEY_SCALE)) return NOVA_KV_OK;
  if (!k_scales) return fail(NOVA_KV_ERR_INVALID_ARG, "k_scales is NULL in the key-scale format");
  if (!aligned(k_scales, 2)) return fail(NOVA_KV_ERR_INVALID_ARG, "k_scales must be 2-byte aligned");
  return NOVA_KV_OK;
}

// The sink-plus-recent band (NULL: none).
nova_kv_status check_band(const nova_kv_band *band) {
  if (!band) return NOVA_KV_OK;
  if (band->n_sink < 0 || band->n_rec < 0) return fail(NOVA_KV_ERR_INVALID_ARG, "band sizes must be >= 0");
  const long long nb = static_cast<long long>(band->n_sink) + band->n_rec;
  if (nb < 1 || nb > NOVA_KV_MAX_BAND)
    return fail(NOVA_KV_ERR_INVALID_ARG, "band of %lld positions (1 .. %d)", nb, NOVA_KV_MAX_BAND);
  if (!band->k || !band->v) return fail(NOVA_KV_ERR_INVALID_ARG, "band k or v is NULL");
  if (!aligned(band->k, 16) || !aligned(band->v, 16))
    return fail(NOVA_KV_ERR_INVALID_ARG, "band buffers must be 16-byte aligned");
  return NOVA_KV_OK;
}

// The (scale, offset) pool of the scalar value arm (ignored otherwise).
nova_kv_status check_sq(const nova_kv_params *p, const void *v_sq) {
  if (!(p->flags & NOVA_KV_SQ_VALUES)) return NOVA_KV_OK;
  if (!v_sq) return fail(NOVA_KV_ERR_INVALID_ARG, "v_sq is NULL in the scalar value format");
  if (!aligned(v_sq, 4)) return fail(NOVA_KV_ERR_INVALID_ARG, "v_sq must be 4-byte aligned");
  return NOVA_KV_OK;
}


namespace {

long long capacity_of(const nova_kv_layout *lay) {
  return static_cast<long long>(lay->block_size) * lay->blocks_per_seq;
}

}  // namespace

nova_kv_status check_metadata(const nova_kv_layout *lay, int32_t num_blocks, int32_t batch,
                              const int32_t *seq_lens, int32_t max_seq_len, const int32_t *start_pos,
                              int32_t n_new) {
  nova_kv_status st = check_layout(lay);
  if (st != NOVA_KV_OK) return st;
  if (batch < 0 || n_new < 0) return fail(NOVA_KV_ERR_INVALID_ARG, "batch and n_new must be >= 0");
  const long long cap = capacity_of(lay);
  if (seq_lens && (max_seq_len < 0 || max_seq_len > cap))
    return fail(NOVA_KV_ERR_INVALID_ARG, "max_seq_len %d outside [0, %lld]", max_seq_len, cap);
  const bool step_write = !start_pos && seq_lens && n_new == 1;
  if (!start_pos && !step_write && n_new > 0)
    return fail(NOVA_KV_ERR_INVALID_ARG, "writes need start_pos (or seq_lens with n_new == 1)");
  const int bs = lay->block_size, bps = lay->blocks_per_seq;
  // physical block of logical block blk of sequence b, or a failure
  auto phys_of = [&](int b, long long blk, long long *phys) -> nova_kv_status {
    if (blk < 0 || blk >= bps)
      return fail(NOVA_KV_ERR_INVALID_ARG, "sequence %d: block %lld outside [0, %d)", b, blk, bps);
    const long long logical = static_cast<long long>(b) * bps + blk;
    const long long p = lay->block_table ? lay->block_table[logical] : logical;
    if (p < 0 || (num_blocks > 0 && p >= num_blocks))
      return fail(NOVA_KV_ERR_INVALID_ARG, "sequence %d: block %lld maps to physical block %lld outside [0, %d)", b,
                  blk, p, num_blocks > 0 ? num_blocks : 0x7fffffff);
    *phys = p;
    return NOVA_KV_OK;
  };
  if (seq_lens) {
    for (int b = 0; b < batch; ++b)
      if (seq_lens[b] < 0 || seq_lens[b] > max_seq_len)
        return fail(NOVA_KV_ERR_INVALID_ARG, "seq_lens[%d] = %d outside [0, max_seq_len = %d]", b, seq_lens[b],
                    max_seq_len);
  }
  // written rows: physical row -> sequence, and physical blocks written
  std::unordered_map<long long, int> row_writer;
  std::unordered_map<long long, int> block_writer;
  for (int b = 0; b < batch; ++b) {
    long long w0 = 0, w1 = 0;  // written positions [w0, w1)
    if (start_pos) {
      w0 = start_pos[b];
      w1 = w0 + n_new;
      if (n_new > 0 && (w0 < 0 || w1 > cap))
        return fail(NOVA_KV_ERR_INVALID_ARG, "sequence %d writes positions [%lld, %lld) outside [0, %lld)", b, w0,
                    w1, cap);
    } else if (step_write && seq_lens[b] > 0) {
      w0 = seq_lens[b] - 1;
      w1 = seq_lens[b];
    }
    for (long long t = w0; t < w1; ++t) {
      long long p = 0;
      if ((st = phys_of(b, t / bs, &p)) != NOVA_KV_OK) return st;
      const long long row = p * bs + t % bs;
      auto it = row_writer.emplace(row, b);
      if (!it.second)
        return fail(NOVA_KV_ERR_INVALID_ARG, "sequences %d and %d write the same row (physical block %lld, row %lld)",
                    it.first->second, b, p, t % bs);
      auto bw = block_writer.emplace(p, b);
      if (!bw.second && bw.first->second != b) bw.first->second = -1;  // written by several sequences
    }
  }
  if (seq_lens) {
    for (int b = 0; b < batch; ++b) {
      const int s = seq_lens[b];
      // every block read must map into the pool and must not be written by
      // another sequence in the same call
      const long long nblk = (static_cast<long long>(s) + bs - 1) / bs;
      for (long long blk = 0; blk < nblk; ++blk) {
        long long p = 0;
        if ((st = phys_of(b, blk, &p)) != NOVA_KV_OK) return st;
        auto it = block_writer.find(p);
        if (it != block_writer.end() && it->second != b)
          return fail(NOVA_KV_ERR_INVALID_ARG,
                      "sequence %d reads physical block %lld, which another sequence writes in the same call", b, p);
      }
    }
  }
  return ok();
}

namespace {

int32_t env_debug() {
  const char *e = getenv("NOVA_KV_DEBUG");
  return e && atoi(e) != 0 ? 1 : 0;
}

std::atomic<int32_t> g_debug{env_debug()};
std::atomic<int32_t> g_debug_blocks{0};

}  // namespace

bool debug_enabled() { return g_debug.load(std::memory_order_relaxed) != 0; }
int32_t debug_num_blocks() { return g_debug_blocks.load(std::memory_order_relaxed); }

}  // namespace host
}  // namespace novakv

using namespace novakv::host;

extern "C" {

const char *nova_kv_status_string(nova_kv_status s) {
  switch (s) {
    case NOVA_KV_OK: return "ok";
    case NOVA_KV_ERR_INVALID_ARG: return "invalid argument";
    case NOVA_KV_ERR_UNSUPPORTED: return "unsupported configuration";
    case NOVA_KV_ERR_WORKSPACE: return "workspace missing or too small";
    case NOVA_KV_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char *nova_kv_last_error(void) { return g_last_error.c_str(); }

nova_kv_status nova_kv_check_metadata(const nova_kv_layout *layout, int32_t num_blocks, int32_t batch,
                                      const int32_t *seq_lens, int32_t max_seq_len, const int32_t *start_pos,
                                      int32_t n_new) {
  return check_metadata(layout, num_blocks, batch, seq_lens, max_seq_len, start_pos, n_new);
}

void nova_kv_set_debug(int32_t on, int32_t num_blocks) {
  g_debug_blocks.store(num_blocks, std::memory_order_relaxed);
  g_debug.store(on ? 1 : 0, std::memory_order_relaxed);
}

}  // extern "C"
