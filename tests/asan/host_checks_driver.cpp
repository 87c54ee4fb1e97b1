// Host program for the sanitizer test of the C ABI's host checks: built with
// AddressSanitizer and UndefinedBehaviorSanitizer together with
// host_checks.cpp.  It runs fixed cases of the argument checks, then reads
// metadata cases from stdin and prints the status of each.
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "../../paper_2608_04074_amd/csrc/host_checks.h"

using namespace novakv::host;

static int expect(const char *what, nova_kv_status got, nova_kv_status want) {
  if (got != want) {
    fprintf(stderr, "%s: status %d, expected %d (%s)\n", what, got, want, nova_kv_last_error());
    return 1;
  }
  return 0;
}

static int fixed_cases() {
  int bad = 0;
  alignas(16) static unsigned char buf[4096];
  nova_kv_params p{};
  p.num_kv_heads = 8;
  p.head_dim = 128;
  p.group_dim = 4;
  p.codebook_size = 256;
  p.kbar = reinterpret_cast<const float *>(buf);
  p.t_k = p.t_k_inv_t = p.t_v = reinterpret_cast<const float *>(buf + 256);
  p.cb_k = p.cb_v = buf + 512;
  bad += expect("params ok", check_params(&p, true, true), NOVA_KV_OK);
  bad += expect("params null", check_params(nullptr, true, true), NOVA_KV_ERR_INVALID_ARG);
  nova_kv_params q = p;
  q.head_dim = 96;
  bad += expect("head_dim 96", check_params(&q, true, true), NOVA_KV_ERR_UNSUPPORTED);
  q = p;
  q.cb_k = buf + 513;
  bad += expect("misaligned codebook", check_params(&q, true, true), NOVA_KV_ERR_INVALID_ARG);
  q = p;
  q.flags = 64;
  bad += expect("unknown flag", check_params(&q, false, true), NOVA_KV_ERR_UNSUPPORTED);
  nova_kv_layout lay{16, 4, nullptr};
  bad += expect("layout ok", check_layout(&lay), NOVA_KV_OK);
  nova_kv_layout big{1 << 16, 1 << 16, nullptr};
  bad += expect("layout too large", check_layout(&big), NOVA_KV_ERR_INVALID_ARG);
  bad += expect("layout null", check_layout(nullptr), NOVA_KV_ERR_INVALID_ARG);
  nova_kv_band band{64, 256, reinterpret_cast<uint16_t *>(buf), reinterpret_cast<uint16_t *>(buf + 16)};
  bad += expect("band ok", check_band(&band), NOVA_KV_OK);
  band.n_rec = 100000;
  bad += expect("band too long", check_band(&band), NOVA_KV_ERR_INVALID_ARG);
  nova_kv_params ks = p;
  ks.flags = NOVA_KV_KEY_SCALE;
  bad += expect("scales missing", check_scales(&ks, nullptr), NOVA_KV_ERR_INVALID_ARG);
  bad += expect("scales odd", check_scales(&ks, buf + 1), NOVA_KV_ERR_INVALID_ARG);
  nova_kv_params sq = p;
  sq.flags = NOVA_KV_SQ_VALUES;
  bad += expect("sq pool missing", check_sq(&sq, nullptr), NOVA_KV_ERR_INVALID_ARG);
  // a long error detail is cut, not overrun
  std::vector<int32_t> lens(3, 1 << 30);
  bad += expect("huge length", check_metadata(&lay, 0, 3, lens.data(), 64, nullptr, 0), NOVA_KV_ERR_INVALID_ARG);
  // epochs: nonzero, distinct, odd for direct calls and even for captured ones
  uint32_t e0 = next_epoch(false), e1 = next_epoch(true), e2 = next_epoch(false), e3 = next_epoch(true);
  if (e0 == 0 || e1 == 0 || e2 == 0 || e3 == 0 || e0 == e2 || e1 == e3 || (e0 & 1) != 1 || (e2 & 1) != 1 ||
      (e1 & 1) != 0 || (e3 & 1) != 0) {
    fprintf(stderr, "epochs %u %u %u %u\n", e0, e1, e2, e3);
    ++bad;
  }
  return bad;
}

static bool read_ints(int n, std::vector<int32_t> &v) {
  v.resize(n > 0 ? n : 0);
  for (int i = 0; i < n; ++i)
    if (scanf("%d", &v[i]) != 1) return false;
  return true;
}

int main() {
  if (fixed_cases() != 0) return 1;
  int ncases = 0;
  if (scanf("%d", &ncases) != 1) return 2;
  for (int c = 0; c < ncases; ++c) {
    int bs, bps, has_table, num_blocks, batch, max_seq, has_seq, has_start, n_new;
    if (scanf("%d %d %d %d %d %d %d %d %d", &bs, &bps, &has_table, &num_blocks, &batch, &max_seq, &has_seq,
              &has_start, &n_new) != 9)
      return 2;
    std::vector<int32_t> table, seq, start;
    if (has_table && !read_ints(batch * bps, table)) return 2;
    if (has_seq && !read_ints(batch, seq)) return 2;
    if (has_start && !read_ints(batch, start)) return 2;
    // exact-size heap arrays, so that a read past any of them is reported
    int32_t *t = has_table ? static_cast<int32_t *>(malloc(sizeof(int32_t) * table.size() + 1)) : nullptr;
    int32_t *s = has_seq ? static_cast<int32_t *>(malloc(sizeof(int32_t) * seq.size() + 1)) : nullptr;
    int32_t *p = has_start ? static_cast<int32_t *>(malloc(sizeof(int32_t) * start.size() + 1)) : nullptr;
    for (size_t i = 0; i < table.size(); ++i) t[i] = table[i];
    for (size_t i = 0; i < seq.size(); ++i) s[i] = seq[i];
    for (size_t i = 0; i < start.size(); ++i) p[i] = start[i];
    nova_kv_layout lay{bs, bps, t};
    const nova_kv_status st = check_metadata(&lay, num_blocks, batch, s, max_seq, p, n_new);
    printf("%d\n", static_cast<int>(st));
    free(t);
    free(s);
    free(p);
  }
  return 0;
}
