// Host-side validation of the C ABI (plain C++, no HIP): argument checks of
// the entry points, the thread-local error detail, and the check of a call's
// device-side metadata (sequence lengths, write positions, block table) on
// host copies, used by nova_kv_check_metadata and by the debug mode.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/nova_kv.h"

namespace novakv {

constexpr int kGroupDim = 4;        // g: coefficients per codebook group
constexpr int kCodebookSize = 256;  // K: codewords per group (8-bit codes)
constexpr int kMaxGqa = 8;          // query heads per KV head handled by the kernels

namespace host {

// Records the detail of a failing call (nova_kv_last_error) and returns s.
nova_kv_status fail(nova_kv_status s, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
// Clears the detail and returns NOVA_KV_OK.
nova_kv_status ok();
bool aligned(const void *p, size_t a);
// Tag of the split exchange of the next decode call: nonzero, new for every
// call; odd for a call launched directly, even for a call captured in a graph.
uint32_t next_epoch(bool captured);

nova_kv_status check_params(const nova_kv_params *p, bool need_encode, bool need_decode);
nova_kv_status check_layout(const nova_kv_layout *lay);
nova_kv_status check_scales(const nova_kv_params *p, const void *k_scales);
nova_kv_status check_band(const nova_kv_band *band);
nova_kv_status check_sq(const nova_kv_params *p, const void *v_sq);

// Host copies of a call's metadata, checked against the layout (see
// nova_kv_check_metadata): block_table is a host array here.
nova_kv_status check_metadata(const nova_kv_layout *lay, int32_t num_blocks, int32_t batch,
                              const int32_t *seq_lens, int32_t max_seq_len, const int32_t *start_pos,
                              int32_t n_new);

// Debug mode (nova_kv_set_debug; initially on when the environment variable
// NOVA_KV_DEBUG is a nonzero number): entry points copy their metadata to
// the host and check it before launching.
bool debug_enabled();
int32_t debug_num_blocks();

}  // namespace host
}  // namespace novakv
