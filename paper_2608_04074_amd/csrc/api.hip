// C ABI of libnovakv: host-side validation, workspace planning and dispatch.
// Every check runs before any HIP call, so an invalid call launches nothing.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/nova_kv.h"
#include "host_checks.h"
#include "nova_kv_internal.h"

using namespace novakv::host;

namespace {

novakv::CacheLayout to_layout(const nova_kv_layout *lay) {
  return novakv::CacheLayout{lay->block_size, lay->blocks_per_seq, lay->block_table};
}

}  // namespace

namespace {

// ---- debug mode: the metadata copied to the host and checked before a launch
nova_kv_status debug_check(const nova_kv_layout *lay, int32_t batch, const int32_t *seq_lens, int32_t max_seq_len,
                           const int32_t *start_pos, int32_t n_new, hipStream_t stream) {
  if (!debug_enabled() || batch <= 0) return NOVA_KV_OK;
  hipError_t e = hipStreamSynchronize(stream);  // the metadata may be written by earlier work on the stream
  auto to_host = [&](const int32_t *d, size_t n, std::vector<int32_t> &h) {
    h.resize(n);
    if (e == hipSuccess) e = hipMemcpy(h.data(), d, n * sizeof(int32_t), hipMemcpyDeviceToHost);
  };
  std::vector<int32_t> lens, starts, table;
  if (seq_lens) to_host(seq_lens, batch, lens);
  if (start_pos) to_host(start_pos, batch, starts);
  if (lay->block_table) to_host(lay->block_table, static_cast<size_t>(batch) * lay->blocks_per_seq, table);
  if (e != hipSuccess) return fail(NOVA_KV_ERR_HIP, "debug mode: metadata copy: %s", hipGetErrorString(e));
  nova_kv_layout hl = *lay;
  hl.block_table = lay->block_table ? table.data() : nullptr;
  const nova_kv_status st = check_metadata(&hl, debug_num_blocks(), batch, seq_lens ? lens.data() : nullptr,
                                           max_seq_len, start_pos ? starts.data() : nullptr, n_new);
  if (st != NOVA_KV_OK) {
    std::string d = "debug mode: ";
    d += nova_kv_last_error();
    return fail(st, "%s", d.c_str());
  }
  return NOVA_KV_OK;
}

// ---- the allocation-free step: a fixed scratch array per GPU
//
// The array's name is a host-side stand-in: host code uses the device address
// that hipGetSymbolAddress returns for the current device (each GPU holds its
// own copy), never the name itself.
constexpr size_t kStaticScratchBytes = NOVA_KV_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

__global__ void fill_zero(uint4 *p, size_t n) {
  for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < n;
       i += static_cast<size_t>(gridDim.x) * blockDim.x)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

// Address of the current device's scratch array; on the first call on a
// device it is looked up and zero-filled by a kernel on `stream` (ordered
// before the caller's launches on that stream).
nova_kv_status static_scratch(hipStream_t stream, void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(NOVA_KV_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(NOVA_KV_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(NOVA_KV_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    fill_zero<<<1024, 256, 0, stream>>>(static_cast<uint4 *>(ptr), kStaticScratchBytes / sizeof(uint4));
    e = hipGetLastError();
    if (e != hipSuccess) return fail(NOVA_KV_ERR_HIP, "scratch clear: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return NOVA_KV_OK;
}

}  // namespace

extern "C" {

nova_kv_status nova_kv_encode(const nova_kv_params *p, const nova_kv_layout *layout,
                              const void *k, const void *v, nova_kv_dtype in_dtype,
                              int32_t batch, int32_t n_new, const int32_t *start_pos,
                              uint8_t *k_codes, uint8_t *v_codes, uint16_t *k_scales,
                              uint16_t *v_sq, const nova_kv_band *band, void *hip_stream) {
  nova_kv_status st = check_params(p, true, false);
  if (st != NOVA_KV_OK) return st;
  if ((st = check_layout(layout)) != NOVA_KV_OK) return st;
  if (batch < 0 || n_new < 0) return fail(NOVA_KV_ERR_INVALID_ARG, "batch and n_new must be >= 0");
  if (in_dtype != NOVA_KV_F32 && in_dtype != NOVA_KV_BF16)
    return fail(NOVA_KV_ERR_INVALID_ARG, "in_dtype must be NOVA_KV_F32 or NOVA_KV_BF16");
  if (batch > 65535) return fail(NOVA_KV_ERR_INVALID_ARG, "batch > 65535");
  if (static_cast<long long>(n_new) > static_cast<long long>(layout->block_size) * layout->blocks_per_seq)
    return fail(NOVA_KV_ERR_INVALID_ARG, "n_new exceeds the per-sequence capacity");
  if (batch == 0 || n_new == 0) return ok();
  if ((st = check_scales(p, k_scales)) != NOVA_KV_OK) return st;
  if ((st = check_sq(p, v_sq)) != NOVA_KV_OK) return st;
  if ((st = check_band(band)) != NOVA_KV_OK) return st;
  if (!k || !v || !start_pos || !k_codes || !v_codes)
    return fail(NOVA_KV_ERR_INVALID_ARG, "k, v, start_pos, k_codes or v_codes is NULL");
  if ((st = debug_check(layout, batch, nullptr, 0, start_pos, n_new, static_cast<hipStream_t>(hip_stream))) !=
      NOVA_KV_OK)
    return st;

  novakv::EncodeArgs a{};
  a.batch = batch;
  a.n_new = n_new;
  a.num_kv_heads = p->num_kv_heads;
  a.head_dim = p->head_dim;
  a.kbar = p->kbar;
  a.t_k = p->t_k;
  a.t_v = p->t_v;
  a.t_bf16 = (p->flags & NOVA_KV_BF16_TRANSFORMS) ? 1 : 0;
  a.cb_k = p->cb_k;
  a.cb_v = p->cb_v;
  a.cb_fp8 = (p->flags & NOVA_KV_FP8_CODEBOOKS) ? 1 : 0;
  a.layout = to_layout(layout);
  a.k = k;
  a.v = v;
  a.in_bf16 = in_dtype == NOVA_KV_BF16;
  a.start_pos = start_pos;
  a.k_codes = k_codes;
  a.v_codes = v_codes;
  a.k_scales = (p->flags & NOVA_KV_KEY_SCALE) ? k_scales : nullptr;
  a.v_sq = (p->flags & NOVA_KV_SQ_VALUES) ? v_sq : nullptr;
  if (band) {
    a.n_sink = band->n_sink;
    a.n_rec = band->n_rec;
    a.band_k = band->k;
    a.band_v = band->v;
  }
  hipError_t e = novakv::launch_encode(a, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return fail(NOVA_KV_ERR_HIP, "encode launch: %s", hipGetErrorString(e));
  return ok();
}

size_t nova_kv_decode_workspace_bytes(const nova_kv_params *p, int32_t batch, int32_t num_q_heads,
                                      int32_t max_seq_len) {
  if (!p || batch <= 0 || num_q_heads <= 0 || max_seq_len <= 0 || p->num_kv_heads <= 0 ||
      p->head_dim <= 0)
    return 0;
  return novakv::plan_decode(batch, num_q_heads, p->num_kv_heads, p->head_dim, max_seq_len, 0, 0).total;
}

namespace {

// Host checks and argument set-up shared by the decode entry points.
nova_kv_status prepare_decode(const nova_kv_params *p, const nova_kv_layout *layout, const void *q,
                              nova_kv_dtype q_dtype, int32_t batch, int32_t num_q_heads, const uint8_t *k_codes,
                              const uint8_t *v_codes, const uint16_t *k_scales, const uint16_t *v_sq,
                              const nova_kv_band *band, const int32_t *seq_lens, int32_t max_seq_len,
                              int32_t window, const float *sinks, float softmax_scale, float *out,
                              void *workspace, size_t workspace_bytes, bool need_encode,
                              novakv::DecodeArgs &a, novakv::DecodePlan &plan,
                              bool static_ws, hipStream_t stream) {
  nova_kv_status st = check_params(p, need_encode, true);
  if (st != NOVA_KV_OK) return st;
  if ((st = check_layout(layout)) != NOVA_KV_OK) return st;
  if (batch < 0) return fail(NOVA_KV_ERR_INVALID_ARG, "batch must be >= 0");
  if (batch > 65535) return fail(NOVA_KV_ERR_INVALID_ARG, "batch > 65535");
  if (num_q_heads <= 0 || num_q_heads % p->num_kv_heads != 0)
    return fail(NOVA_KV_ERR_INVALID_ARG, "num_q_heads (%d) must be a positive multiple of num_kv_heads (%d)",
                num_q_heads, p->num_kv_heads);
  if (num_q_heads / p->num_kv_heads > novakv::kMaxGqa)
    return fail(NOVA_KV_ERR_UNSUPPORTED, "more than %d query heads per KV head", novakv::kMaxGqa);
  if (max_seq_len <= 0) return fail(NOVA_KV_ERR_INVALID_ARG, "max_seq_len must be > 0");
  if (static_cast<long long>(max_seq_len) > static_cast<long long>(layout->block_size) * layout->blocks_per_seq)
    return fail(NOVA_KV_ERR_INVALID_ARG, "max_seq_len exceeds the per-sequence capacity");
  if (window < 0) return fail(NOVA_KV_ERR_INVALID_ARG, "window must be >= 0");
  if (q_dtype != NOVA_KV_F32 && q_dtype != NOVA_KV_BF16)
    return fail(NOVA_KV_ERR_INVALID_ARG, "q_dtype must be NOVA_KV_F32 or NOVA_KV_BF16");
  if (!(softmax_scale >= 0.f)) return fail(NOVA_KV_ERR_INVALID_ARG, "softmax_scale must be >= 0");
  if (batch == 0) return NOVA_KV_OK;
  if ((st = check_scales(p, k_scales)) != NOVA_KV_OK) return st;
  if ((st = check_sq(p, v_sq)) != NOVA_KV_OK) return st;
  if ((st = check_band(band)) != NOVA_KV_OK) return st;
  if (!q || !k_codes || !v_codes || !seq_lens || !out)
    return fail(NOVA_KV_ERR_INVALID_ARG, "q, k_codes, v_codes, seq_lens or out is NULL");
  if (!aligned(k_codes, 16) || !aligned(v_codes, 16))
    return fail(NOVA_KV_ERR_INVALID_ARG, "code pools must be 16-byte aligned");
  // every value format runs on the table kernels where their layout applies
  const bool sq = (p->flags & NOVA_KV_SQ_VALUES) != 0;
  plan = novakv::plan_decode(batch, num_q_heads, p->num_kv_heads, p->head_dim, max_seq_len, layout->block_size,
                             window, false);
  if ((st = debug_check(layout, batch, seq_lens, max_seq_len, nullptr, need_encode ? 1 : 0, stream)) != NOVA_KV_OK)
    return st;
  if (static_ws) {  // the allocation-free step: the GPU's fixed scratch array (the last check)
    if (plan.total > kStaticScratchBytes)
      return fail(NOVA_KV_ERR_WORKSPACE,
                  "this shape needs %zu bytes of scratch; the allocation-free step holds %zu "
                  "(call nova_kv_append_decode_attn with a workspace)",
                  plan.total, kStaticScratchBytes);
    if ((st = static_scratch(stream, &workspace)) != NOVA_KV_OK) return st;
    workspace_bytes = kStaticScratchBytes;
  }
  if (!workspace || workspace_bytes < plan.total)
    return fail(NOVA_KV_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", plan.total,
                workspace ? workspace_bytes : static_cast<size_t>(0));
  if (!aligned(workspace, 256)) return fail(NOVA_KV_ERR_WORKSPACE, "workspace must be 256-byte aligned");

  a = novakv::DecodeArgs{};
  a.batch = batch;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = p->num_kv_heads;
  a.head_dim = p->head_dim;
  a.gqa = num_q_heads / p->num_kv_heads;
  a.kbar = p->kbar;
  a.t_k_inv_t = p->t_k_inv_t;
  a.t_v = p->t_v;
  a.t_bf16 = (p->flags & NOVA_KV_BF16_TRANSFORMS) ? 1 : 0;
  a.cb_k = p->cb_k;
  a.cb_v = p->cb_v;
  a.cb_fp8 = (p->flags & NOVA_KV_FP8_CODEBOOKS) ? 1 : 0;
  a.layout = to_layout(layout);
  a.q = q;
  a.q_bf16 = q_dtype == NOVA_KV_BF16;
  a.k_codes = k_codes;
  a.v_codes = v_codes;
  a.k_scales = (p->flags & NOVA_KV_KEY_SCALE) ? k_scales : nullptr;
  a.v_sq = sq ? v_sq : nullptr;
  if (band) {
    a.n_sink = band->n_sink;
    a.n_rec = band->n_rec;
    a.band_k = band->k;
    a.band_v = band->v;
  }
  a.seq_lens = seq_lens;
  a.max_seq_len = max_seq_len;
  a.window = window;
  a.sinks = sinks;
  a.scale = softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf(static_cast<float>(p->head_dim));
  a.qscale = plan.use_lut ? a.scale * 1.44269504088896341f : a.scale;
  a.out = out;
  char *ws = static_cast<char *>(workspace);
  a.counters = reinterpret_cast<int *>(ws + plan.off_cnt);
  a.qp = reinterpret_cast<float *>(ws + plan.off_qp);
  a.sinkp = reinterpret_cast<float *>(ws + plan.off_sinkp);
  a.part_ml = reinterpret_cast<float *>(ws + plan.off_ml);
  a.part_acc = reinterpret_cast<float *>(ws + plan.off_acc);
  a.newp = reinterpret_cast<float *>(ws + plan.off_new);
  a.xch = reinterpret_cast<uint64_t *>(ws + plan.off_xch);
  a.xnew = reinterpret_cast<uint64_t *>(ws + plan.off_xnew);
  a.n_split = plan.n_split;
  a.chunk = plan.chunk;
  a.b_chunk = novakv::plan_b_chunk(batch, p->num_kv_heads, plan.n_split);
  a.xgrp = reinterpret_cast<uint64_t *>(ws + plan.off_xgrp);
  a.group_size = plan.n_split;
  a.n_group = 1;
  if (plan.use_lut && p->head_dim == 128) {
    a.group_size = novakv::plan_group_size(plan.n_split);
    a.n_group = (plan.n_split + a.group_size - 1) / a.group_size;
  }
  // A call captured in a graph is replayed with these arguments, its epoch
  // included, so its readers empty the exchange words they read.
  hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &capture) != hipSuccess) {
    (void)hipGetLastError();
    capture = hipStreamCaptureStatusNone;
  }
  a.clear_xch = capture == hipStreamCaptureStatusActive ? 1 : 0;
  a.epoch = next_epoch(a.clear_xch != 0);
  return NOVA_KV_OK;
}

}  // namespace

nova_kv_status nova_kv_decode_attn(const nova_kv_params *p, const nova_kv_layout *layout,
                                   const void *q, nova_kv_dtype q_dtype, int32_t batch,
                                   int32_t num_q_heads, const uint8_t *k_codes,
                                   const uint8_t *v_codes, const uint16_t *k_scales, const uint16_t *v_sq,
                                   const nova_kv_band *band, const int32_t *seq_lens, int32_t max_seq_len,
                                   int32_t window, const float *sinks,
                                   float softmax_scale, float *out, void *workspace,
                                   size_t workspace_bytes, void *hip_stream) {
  novakv::DecodeArgs a;
  novakv::DecodePlan plan;
  nova_kv_status st = prepare_decode(p, layout, q, q_dtype, batch, num_q_heads, k_codes, v_codes, k_scales, v_sq,
                                     band, seq_lens, max_seq_len, window, sinks, softmax_scale, out, workspace, workspace_bytes,
                                     false, a, plan, false, static_cast<hipStream_t>(hip_stream));
  if (st != NOVA_KV_OK || batch == 0) return st == NOVA_KV_OK ? ok() : st;
  hipError_t e = novakv::launch_decode(a, plan.use_lut, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return fail(NOVA_KV_ERR_HIP, "decode launch: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"

namespace {

// The step of nova_kv_append_decode_attn, with the caller's workspace or
// (static_ws) the GPU's fixed scratch array.
nova_kv_status append_step(const nova_kv_params *p, const nova_kv_layout *layout, const void *k_new,
                           const void *v_new, nova_kv_dtype new_dtype, const void *q, nova_kv_dtype q_dtype,
                           int32_t batch, int32_t num_q_heads, uint8_t *k_codes, uint8_t *v_codes,
                           uint16_t *k_scales, uint16_t *v_sq, const nova_kv_band *band, const int32_t *seq_lens,
                           int32_t max_seq_len, int32_t window, const float *sinks, float softmax_scale, float *out,
                           void *workspace, size_t workspace_bytes, bool static_ws, void *hip_stream) {
  if (new_dtype != NOVA_KV_F32 && new_dtype != NOVA_KV_BF16)
    return fail(NOVA_KV_ERR_INVALID_ARG, "new_dtype must be NOVA_KV_F32 or NOVA_KV_BF16");
  if (batch > 0 && (!k_new || !v_new)) return fail(NOVA_KV_ERR_INVALID_ARG, "k_new or v_new is NULL");
  const hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  novakv::DecodeArgs a;
  novakv::DecodePlan plan;
  nova_kv_status st = prepare_decode(p, layout, q, q_dtype, batch, num_q_heads, k_codes, v_codes, k_scales,
                                     v_sq, band, seq_lens, max_seq_len, window, sinks, softmax_scale, out, workspace,
                                     workspace_bytes, true, a, plan, static_ws, stream);
  if (st != NOVA_KV_OK || batch == 0) return st == NOVA_KV_OK ? ok() : st;
  hipError_t e;
  // One launch on a table kernel.  With a band whose recent part holds the
  // new token, in any format and at either head_dim, that token is the band's
  // last row; otherwise (head_dim 128, plain or fp8 codebooks) it is attended
  // from its codes, which the splits of a (sequence, KV head) encode between
  // them: with one split, one workgroup's encoder team would encode all 8
  // blocks while its token loop runs, and two launches are faster (B = 32,
  // S = 32K: paged 133 us against 171 us in one launch).  The head_dim-128
  // band step on a paged cache with one split per unit also runs as encode
  // then decode (deployed format, B = 32, S = 32K: 166 us against 189 us in
  // one launch; on a contiguous cache the one launch stays as fast).
  const bool scaled_format = (p->flags & (NOVA_KV_KEY_SCALE | NOVA_KV_SQ_VALUES)) != 0;
  const bool fused =
      plan.use_lut && (band ? band->n_rec >= 1 && (plan.n_split > 1 || !layout->block_table || p->head_dim != 128)
                            : p->head_dim == 128 && !scaled_format && plan.n_split > 1);
  if (fused) {
    a.append = 1;
    a.k_new = k_new;
    a.v_new = v_new;
    a.new_bf16 = new_dtype == NOVA_KV_BF16;
    a.t_k = p->t_k;
    a.k_codes_w = k_codes;
    a.v_codes_w = v_codes;
    a.k_scales_w = (p->flags & NOVA_KV_KEY_SCALE) ? k_scales : nullptr;
    a.v_sq_w = (p->flags & NOVA_KV_SQ_VALUES) ? v_sq : nullptr;
    if (band) {
      a.band_k_w = static_cast<uint16_t *>(band->k);
      a.band_v_w = static_cast<uint16_t *>(band->v);
    }
    e = novakv::launch_decode(a, plan.use_lut, stream);
  } else {
    // the one-token encode at position seq_lens[b] - 1, then the decode
    novakv::EncodeArgs ea{};
    ea.batch = batch;
    ea.n_new = 1;
    ea.num_kv_heads = p->num_kv_heads;
    ea.head_dim = p->head_dim;
    ea.kbar = p->kbar;
    ea.t_k = p->t_k;
    ea.t_v = p->t_v;
    ea.t_bf16 = (p->flags & NOVA_KV_BF16_TRANSFORMS) ? 1 : 0;
    ea.cb_k = p->cb_k;
    ea.cb_v = p->cb_v;
    ea.cb_fp8 = (p->flags & NOVA_KV_FP8_CODEBOOKS) ? 1 : 0;
    ea.layout = to_layout(layout);
    ea.k = k_new;
    ea.v = v_new;
    ea.in_bf16 = new_dtype == NOVA_KV_BF16;
    ea.start_pos = seq_lens;
    ea.start_offset = -1;
    ea.k_codes = k_codes;
    ea.v_codes = v_codes;
    ea.k_scales = (p->flags & NOVA_KV_KEY_SCALE) ? k_scales : nullptr;
    ea.v_sq = (p->flags & NOVA_KV_SQ_VALUES) ? v_sq : nullptr;
    if (band) {
      ea.n_sink = band->n_sink;
      ea.n_rec = band->n_rec;
      ea.band_k = band->k;
      ea.band_v = band->v;
    }
    e = novakv::launch_encode(ea, stream);
    if (e == hipSuccess) e = novakv::launch_decode(a, plan.use_lut, stream);
  }
  if (e != hipSuccess) return fail(NOVA_KV_ERR_HIP, "append-decode launch: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

nova_kv_status nova_kv_append_decode_attn(const nova_kv_params *p, const nova_kv_layout *layout,
                                          const void *k_new, const void *v_new, nova_kv_dtype new_dtype,
                                          const void *q, nova_kv_dtype q_dtype, int32_t batch,
                                          int32_t num_q_heads, uint8_t *k_codes, uint8_t *v_codes,
                                          uint16_t *k_scales, uint16_t *v_sq, const nova_kv_band *band,
                                          const int32_t *seq_lens, int32_t max_seq_len,
                                          int32_t window,
                                          const float *sinks, float softmax_scale, float *out,
                                          void *workspace, size_t workspace_bytes, void *hip_stream) {
  return append_step(p, layout, k_new, v_new, new_dtype, q, q_dtype, batch, num_q_heads, k_codes, v_codes,
                     k_scales, v_sq, band, seq_lens, max_seq_len, window, sinks, softmax_scale, out, workspace,
                     workspace_bytes, false, hip_stream);
}

nova_kv_status nova_kv_append_decode_attn_noalloc(const nova_kv_params *p, const nova_kv_layout *layout,
                                                  const void *k_new, const void *v_new, nova_kv_dtype new_dtype,
                                                  const void *q, nova_kv_dtype q_dtype, int32_t batch,
                                                  int32_t num_q_heads, uint8_t *k_codes, uint8_t *v_codes,
                                                  uint16_t *k_scales, uint16_t *v_sq, const nova_kv_band *band,
                                                  const int32_t *seq_lens, int32_t max_seq_len, int32_t window,
                                                  const float *sinks, float softmax_scale, float *out,
                                                  void *hip_stream) {
  return append_step(p, layout, k_new, v_new, new_dtype, q, q_dtype, batch, num_q_heads, k_codes, v_codes,
                     k_scales, v_sq, band, seq_lens, max_seq_len, window, sinks, softmax_scale, out, nullptr, 0,
                     true, hip_stream);
}

}  // extern "C"
