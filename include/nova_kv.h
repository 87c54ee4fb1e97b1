/*
 * nova_kv.h -- C ABI of the NOVA-KV hot path on MI355X (gfx950).
 *
 * NOVA-KV ("Spend Bits Where Queries Look: KV Cache Vector Quantization with
 * Attention-Preserving Transforms") stores every cached key and value as one
 * 8-bit codebook index per group of g = 4 transform coefficients, i.e. 2 bits
 * per element.  This library implements the calls a serving engine makes on
 * that cache:
 *
 *   nova_kv_encode       append-time write path: transform the new keys and
 *                        values, pick the nearest codeword of every group, and
 *                        store the code bytes (paper: Algorithm 1, "Write";
 *                        Theorem 1 and Corollary 1 for the transforms; Sec.
 *                        "Calibration": the codeword at the smallest squared
 *                        distance, searched over the whole codebook).
 *   nova_kv_decode_attn  single-token decode attention read straight from the
 *                        codes (paper: Algorithm 1, "Attention"; Sec. "Decoding
 *                        kernel and read path"; Appendix "Attention sinks in the
 *                        quantized serving path").
 *   nova_kv_append_decode_attn  both for one decode step (append the step's
 *                        token, then attend), in a single launch where the
 *                        shape allows.
 *
 * Conventions for every call
 *   - All tensor pointers are DEVICE pointers owned by the caller; the library
 *     never allocates, frees or synchronizes inside these calls.  All work is
 *     enqueued on `hip_stream` (a hipStream_t passed as void*; NULL = default
 *     stream) and completes asynchronously.
 *   - Structs are passed by host pointer and read only during the call.
 *   - Arguments are validated on the host before anything is launched; on any
 *     error nothing is launched and a status != NOVA_KV_OK is returned, with a
 *     human-readable detail in nova_kv_last_error() (thread-local).
 *   - Device-resident values (seq_lens, start_pos, block_table entries) cannot
 *     be checked without a synchronisation; their preconditions are stated
 *     per call and are the caller's responsibility.
 *   - All arrays are dense and row-major in the index order written.
 */
#ifndef NOVA_KV_H
#define NOVA_KV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    NOVA_KV_OK = 0,
    NOVA_KV_ERR_INVALID_ARG = 1,   /* NULL required pointer, bad shape or count   */
    NOVA_KV_ERR_UNSUPPORTED = 2,   /* valid but not implemented (g != 4, D, flags) */
    NOVA_KV_ERR_WORKSPACE = 3,     /* workspace missing or too small               */
    NOVA_KV_ERR_HIP = 4            /* a HIP runtime call or kernel launch failed   */
} nova_kv_status;

typedef enum {
    NOVA_KV_F32 = 0,               /* IEEE fp32                                    */
    NOVA_KV_BF16 = 1               /* bfloat16, stored as uint16 bit patterns      */
} nova_kv_dtype;

/*
 * Per-layer calibration outputs (paper: Algorithm 2 and 3; Sec. "Reported
 * quantities" lists what is stored per (layer, KV head)).  Hkv = num_kv_heads,
 * D = head_dim, L = D / group_dim, K = codebook_size.
 *
 *   kbar      [Hkv][D]      fp32  key mean k_bar
 *   t_k       [Hkv][D][D]   fp32 (or bf16, below)  key transform R_K with the
 *                                 grouping folded into its columns:
 *                                 r = (k - k_bar) @ t_k
 *   t_k_inv_t [Hkv][D][D]   R_K^{-T} (same column order): q' = q @ t_k_inv_t
 *   t_v       [Hkv][D][D]   value transform R_V (orthogonal, columns
 *                                 grouped):  s = v @ t_v,  v_hat = s_hat @ t_v^T
 *   cb_k      [Hkv][L][K][g] fp16 bit patterns (uint16), or fp8 E4M3 bytes
 *                           with NOVA_KV_FP8_CODEBOOKS: key codebook of each group
 *   cb_v      [Hkv][L][K][g] the same for the value codebooks
 *
 * Group l covers transform coordinates [l*g, (l+1)*g).  Supported: g = 4,
 * K = 256, D in {64, 128}.  Every array must be 16-byte aligned
 * (NOVA_KV_ERR_INVALID_ARG otherwise).
 *
 *   flags     0 or any combination of the four formats below.
 *             NOVA_KV_KEY_SCALE: the key-scale format (paper: Algorithm
 *             2 normalizes r_j by rho_j = ||r_j||_2 / sqrt(D) before the
 *             codebooks are trained; Sec. "Bit rate": a BF16 scale per token;
 *             Sec. "Decoding kernel and read path": the read path multiplies
 *             the partial logit by it).  cb_k must then hold codebooks of
 *             normalized coefficients, and every call takes a k_scales pool.
 *             NOVA_KV_FP8_CODEBOOKS: the
 *             codebooks are stored as fp8 E4M3 bytes (OCP format: bias 7, no
 *             infinities; paper: Sec. "Calibration", the fp16 codebooks are
 *             rounded to fp8 ahead of use), 4 bytes per codeword; every value
 *             is used exactly (E4M3 values are exact in fp16).
 *             NOVA_KV_SQ_VALUES: the scalar value arm (paper: Sec. "Bit rate"
 *             and the implementation table: per-token affine INT2 values with
 *             a BF16 scale and offset).  A token's values are rotated by t_v
 *             (any orthogonal matrix), s = v @ t_v, and every coordinate is
 *             stored as a 2-bit code q of the grid offset + scale * q, with
 *             offset = bf16(min_i s_i), scale = bf16((max_i s_i - min_i s_i) / 3)
 *             and q_i = clamp(round_half_even((s_i - offset) / scale), 0, 3)
 *             (q = 0 when the stored scale is 0); coordinate 4g + j sits in
 *             bits 2j, 2j+1 of byte g of the token's value code row.  cb_v is
 *             then unused (may be NULL) and every call takes a v_sq pool.
 *             NOVA_KV_BF16_TRANSFORMS: t_k, t_k_inv_t and t_v are bf16 bit
 *             patterns (uint16) instead of fp32 (paper: Sec. "Calibration",
 *             the bases are cast to bfloat16 when loaded into the serving
 *             engine); every kernel reads them as those exact values.
 *             Other bits are reserved (NOVA_KV_ERR_UNSUPPORTED).
 */
#define NOVA_KV_KEY_SCALE 1u
#define NOVA_KV_FP8_CODEBOOKS 2u
#define NOVA_KV_SQ_VALUES 4u
#define NOVA_KV_BF16_TRANSFORMS 8u

typedef struct {
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t group_dim;
    int32_t codebook_size;
    uint32_t flags;
    const float *kbar;
    const void *t_k;        /* fp32, or bf16 bit patterns with NOVA_KV_BF16_TRANSFORMS */
    const void *t_k_inv_t;
    const void *t_v;
    const void *cb_k;
    const void *cb_v;
} nova_kv_params;

/*
 * Code pool layout (paper: the codes go into a fixed-width paged cache,
 * Fig. 2b).  One pool for key codes and one for value codes, each
 *
 *   uint8 codes[num_blocks][Hkv][block_size][L]
 *
 * Token t of sequence b lives in logical block i = t / block_size at row
 * t % block_size of physical block
 *   p = block_table ? block_table[b * blocks_per_seq + i] : b * blocks_per_seq + i.
 *
 * A contiguous cache is block_table = NULL, blocks_per_seq = 1 and
 * block_size = the per-sequence capacity (codes[B][Hkv][capacity][L]).
 * block_table is a DEVICE int32 array [B][blocks_per_seq]; every entry used
 * must index a physical block of both pools (caller's precondition).  Both
 * pools must be 16-byte aligned.
 */
typedef struct {
    int32_t block_size;
    int32_t blocks_per_seq;
    const int32_t *block_table;
} nova_kv_layout;

/*
 * Sink-plus-recent band (paper: Sec. "Sink-plus-recent band" and the figure
 * of the cache layout at decoding position t): the first n_sink and the most
 * recent n_rec positions of every sequence are held in BF16 and attended with
 * their exact keys and values; the positions in between are read from the
 * code pools.  With S cached tokens the band is positions [0, n_sink) and
 * [max(n_sink, S - n_rec), S) (inside the attended range).
 *
 *   n_sink, n_rec  >= 0, n_sink + n_rec in [1, NOVA_KV_MAX_BAND]
 *   k, v      uint16 bf16 bit patterns [B][Hkv][n_sink + n_rec][D], device,
 *             16-byte aligned; b is the sequence index of the call.  Position
 *             p sits in slot p when p < n_sink, else in slot
 *             n_sink + (p mod n_rec) (a ring holding the last n_rec positions).
 *
 * Calls take a `const nova_kv_band *` (NULL = no band).  nova_kv_encode writes
 * the band rows of the new tokens that are in the band once the append is
 * done (p < n_sink, or p >= start_pos[b] + n_new - n_rec) and, as without a
 * band, the codes of every new token, so a position that leaves the recent
 * band is read from codes written when it was appended.  Inputs in fp32 are
 * rounded to bf16 (to nearest even) for the band.
 */
#define NOVA_KV_MAX_BAND 1024

typedef struct {
    int32_t n_sink;
    int32_t n_rec;
    uint16_t *k;
    uint16_t *v;
} nova_kv_band;

/*
 * nova_kv_encode -- append n_new tokens per sequence to the code pools.
 *
 * Paper: Algorithm 1 ("Write": cache Q+((k_j - k_bar) R_K)); Theorem 1
 * (r = (k - k_bar) R_K); Corollary 1 (s = v R_V); Sec. "Calibration"
 * (nearest codeword, Euclidean metric, transform domain).
 *
 *   k, v       [B][n_new][Hkv][D] device, dtype in_dtype (F32 or BF16)
 *   start_pos  [B] int32 device: position of the first new token of each
 *              sequence; precondition start_pos[b] + n_new <= block_size *
 *              blocks_per_seq.  A token whose position falls outside
 *              [0, block_size * blocks_per_seq) is not stored (nothing of it is
 *              written: codes, scales or band rows).
 *   k_codes, v_codes  code pools (see nova_kv_layout), written at positions
 *              start_pos[b] .. start_pos[b] + n_new - 1; nothing else is touched.
 *   k_scales   key-scale format only (else ignored, may be NULL): the scale
 *              pool, uint16 bf16 bit patterns [num_blocks][Hkv][block_size]
 *              addressed like the code pools (one scale per token-head),
 *              2-byte aligned, written at the same positions.
 *   v_sq       scalar value arm only (else ignored, may be NULL): uint16 bf16
 *              bit patterns [num_blocks][Hkv][block_size][2] (scale, offset)
 *              addressed like the code pools, 4-byte aligned, written at the
 *              new positions.
 *   band       NULL, or the sink-plus-recent band: the new tokens that are in
 *              it after the append are also written there (bf16).
 *
 * For every (b, token, KV head, group l) the stored byte is the smallest index
 * c minimising sum_i (u_i - cb[l][c][i])^2, u the group's coefficients; the
 * transform and the distances are evaluated in fp64.  In the key-scale format
 * the key side quantizes u / rho with rho = sqrt(sum of the D squared
 * coefficients, added in coordinate order) / sqrt(D) (u = 0 when rho = 0), and
 * stores rho rounded to fp32 and then to bf16 (each to nearest even).
 * batch == 0 or n_new == 0 is a valid no-op.
 */
nova_kv_status nova_kv_encode(const nova_kv_params *p, const nova_kv_layout *layout,
                              const void *k, const void *v, nova_kv_dtype in_dtype,
                              int32_t batch, int32_t n_new, const int32_t *start_pos,
                              uint8_t *k_codes, uint8_t *v_codes, uint16_t *k_scales,
                              uint16_t *v_sq, const nova_kv_band *band, void *hip_stream);

/*
 * Bytes of device workspace nova_kv_decode_attn needs for this shape (split
 * arrival counters, split partials, pre-transformed queries).  Returns 0 on
 * invalid input.
 */
size_t nova_kv_decode_workspace_bytes(const nova_kv_params *p, int32_t batch,
                                      int32_t num_q_heads, int32_t max_seq_len);

/*
 * nova_kv_decode_attn -- one decode step of attention over the code pools.
 *
 * Paper: Algorithm 1 ("Attention": softmax(Q R_K^{-T} Q-(K_hat)^T / sqrt(d)));
 * Sec. "Decoding kernel and read path" (q R_K^{-T} formed once per step, one
 * codeword lookup per group, k_bar dropped by Lemma S1, two-stage split-KV
 * decode); Corollary 1 (v_hat = s_hat R_V^T); Appendix "Attention sinks"
 * (sink added once after the split combine, shifted by -(q . k_bar) * scale).
 *
 *   q          [B][Hq][D] device, dtype q_dtype (F32 or BF16); query head h
 *              reads KV head h / (Hq / Hkv).
 *   k_scales   key-scale format only (else ignored, may be NULL): the scale
 *              pool of nova_kv_encode, read at the attended positions.
 *   v_sq       scalar value arm only (else ignored, may be NULL): the
 *              (scale, offset) pool of nova_kv_encode.
 *   band       NULL, or the sink-plus-recent band: its attended positions
 *              are read from it (exact bf16 keys and values, key scales
 *              unused), the other attended positions from the pools.
 *   seq_lens   [B] int32 device: cached tokens of each sequence (the current
 *              token already appended); precondition 0 <= seq_lens[b] <= max_seq_len.
 *   max_seq_len  host upper bound of seq_lens; must not exceed the layout's
 *              per-sequence capacity block_size * blocks_per_seq.
 *   window     0 = attend to all seq_lens[b] tokens; W > 0 = the last W only.
 *   sinks      [Hq] fp32 device learned sink logits (scaled-logit units, no
 *              value vector), or NULL.
 *   softmax_scale  logit scale; 0 selects 1/sqrt(D).
 *   out        [B][Hq][D] fp32 device:
 *                out = sum_t p_t v_hat_t,  p = softmax({z_t} U {sink}),
 *                z_t = q . k_hat_t * scale,  k_hat_t = r_hat_t t_k_inv_t^T + k_bar,
 *                v_hat_t = s_hat_t t_v^T;
 *              in the key-scale format r_hat_t is rho_t times the codewords,
 *              rho_t the stored bf16 scale.
 *              A row with no attended token and no sink is written as zeros.
 *   workspace  device scratch of at least nova_kv_decode_workspace_bytes(...)
 *              bytes, 256-byte aligned.  It must be zero-filled before its
 *              first use (e.g. hipMemset once after allocation); every call
 *              leaves it ready for the next one, so it is never cleared again.
 *              This holds for replays of a call captured in a HIP graph too
 *              (they repeat the captured arguments): the words the splits
 *              exchange are emptied by their reader within the call.
 *              Calls that share a workspace must be ordered on one stream.
 * batch == 0 is a valid no-op.
 */
nova_kv_status nova_kv_decode_attn(const nova_kv_params *p, const nova_kv_layout *layout,
                                   const void *q, nova_kv_dtype q_dtype,
                                   int32_t batch, int32_t num_q_heads,
                                   const uint8_t *k_codes, const uint8_t *v_codes,
                                   const uint16_t *k_scales, const uint16_t *v_sq,
                                   const nova_kv_band *band,
                                   const int32_t *seq_lens, int32_t max_seq_len,
                                   int32_t window, const float *sinks, float softmax_scale,
                                   float *out, void *workspace, size_t workspace_bytes,
                                   void *hip_stream);

/*
 * nova_kv_append_decode_attn -- one decode step in one call: append the step's
 * key and value of every sequence to the code pools, then attend over the
 * cache including them.
 *
 * Paper: Algorithm 1 (the "Write" of the new token, then "Attention"; Fig. 2:
 * write, then read), with the references of nova_kv_encode and
 * nova_kv_decode_attn.
 *
 *   k_new, v_new  [B][Hkv][D] device, dtype new_dtype (F32 or BF16): the token
 *              at position seq_lens[b] - 1 of each sequence (the newest cached
 *              token).  A sequence with seq_lens[b] == 0 stores nothing and
 *              attends to nothing: its output rows are zeros.
 *   k_codes, v_codes (and k_scales, v_sq in their formats, band when
 *              given)  written at position seq_lens[b] - 1 exactly as
 *              nova_kv_encode(n_new = 1, start_pos = seq_lens - 1) writes them
 *              (same bytes); nothing else is touched.
 *   all other arguments as in nova_kv_decode_attn (params also need t_k).
 *
 * out equals the output of nova_kv_decode_attn over the pools after that
 * append, up to fp32 rounding.  On 16-aligned blocks the step is a single
 * kernel launch, in which the workgroups that read the pools also encode the
 * new token and store what nova_kv_encode would:
 *   - any format (key scale, scalar value arm, fp8) with a band whose n_rec
 *     >= 1, at head_dim 64, and at head_dim 128 on a contiguous cache or when
 *     the planner splits each (sequence, KV head) over more than one
 *     workgroup: the new token is the band's last row, stored in the launch
 *     and attended exactly from it, as the decode after the encode would;
 *   - head_dim 128, plain or fp8 codebooks, no band, when the planner splits
 *     each (sequence, KV head) over more than one workgroup: the new token
 *     is attended from its codes (its term is added after the split combine
 *     instead of inside a split).
 * Otherwise the one-token encode and the decode run one after the other on
 * the stream.
 * batch == 0 is a valid no-op.
 */
nova_kv_status nova_kv_append_decode_attn(const nova_kv_params *p, const nova_kv_layout *layout,
                                          const void *k_new, const void *v_new, nova_kv_dtype new_dtype,
                                          const void *q, nova_kv_dtype q_dtype,
                                          int32_t batch, int32_t num_q_heads,
                                          uint8_t *k_codes, uint8_t *v_codes, uint16_t *k_scales,
                                          uint16_t *v_sq, const nova_kv_band *band,
                                          const int32_t *seq_lens, int32_t max_seq_len,
                                          int32_t window, const float *sinks, float softmax_scale,
                                          float *out, void *workspace, size_t workspace_bytes,
                                          void *hip_stream);

/*
 * nova_kv_append_decode_attn_noalloc -- nova_kv_append_decode_attn without a
 * workspace argument, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  It allocates nothing: its scratch is a fixed array of
 * NOVA_KV_NOALLOC_SCRATCH_BYTES (32 MiB) in the library's device image, one
 * copy per GPU, held until the process ends.
 *
 *   Arguments, results and written bytes as in nova_kv_append_decode_attn.
 *   A shape whose workspace (nova_kv_decode_workspace_bytes) exceeds the
 *   array is rejected with NOVA_KV_ERR_WORKSPACE before any HIP call.
 *   The first call on a device looks the array up for the current device and
 *   zero-fills it with a kernel on hip_stream, ahead of the step.
 *   Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 *   (on different streams, or from several threads without ordering) race;
 *   order them on one stream.  A call may be captured in a HIP graph and
 *   replayed; make one call outside the capture first, so that the array is
 *   looked up and cleared before the graph runs.
 * batch == 0 is a valid no-op.
 */
#define NOVA_KV_NOALLOC_SCRATCH_BYTES (32u << 20)
nova_kv_status nova_kv_append_decode_attn_noalloc(const nova_kv_params *p, const nova_kv_layout *layout,
                                                  const void *k_new, const void *v_new, nova_kv_dtype new_dtype,
                                                  const void *q, nova_kv_dtype q_dtype,
                                                  int32_t batch, int32_t num_q_heads,
                                                  uint8_t *k_codes, uint8_t *v_codes, uint16_t *k_scales,
                                                  uint16_t *v_sq, const nova_kv_band *band,
                                                  const int32_t *seq_lens, int32_t max_seq_len,
                                                  int32_t window, const float *sinks, float softmax_scale,
                                                  float *out, void *hip_stream);

/*
 * nova_kv_check_metadata -- host-side check of a call's metadata, the
 * preconditions the kernels take on trust.  All pointers are HOST arrays
 * here (layout->block_table included).  Nothing is launched; usable without
 * a GPU.
 *
 *   num_blocks  physical blocks of the pools (> 0), or <= 0 if unknown (then
 *               block-table entries are only checked to be >= 0).
 *   seq_lens    [batch] or NULL: sequences read positions [0, seq_lens[b]);
 *               requires 0 <= seq_lens[b] <= max_seq_len <= capacity.
 *   start_pos   [batch] or NULL: nova_kv_encode writes positions
 *               [start_pos[b], start_pos[b] + n_new), all inside
 *               [0, block_size * blocks_per_seq).  With start_pos NULL,
 *               seq_lens given and n_new == 1, the write of
 *               nova_kv_append_decode_attn: position seq_lens[b] - 1 (none
 *               for an empty sequence).
 * Every logical block holding a read or written position must map to a
 * physical block in [0, num_blocks); no two sequences may write the same
 * row; no sequence may read a physical block that another one writes in the
 * same call.  Returns NOVA_KV_ERR_INVALID_ARG with the first offending entry
 * in nova_kv_last_error(), else NOVA_KV_OK.
 */
nova_kv_status nova_kv_check_metadata(const nova_kv_layout *layout, int32_t num_blocks, int32_t batch,
                                      const int32_t *seq_lens, int32_t max_seq_len, const int32_t *start_pos,
                                      int32_t n_new);

/*
 * nova_kv_set_debug -- debug mode of the entry points (process-wide; also on
 * from the start when the environment variable NOVA_KV_DEBUG is a nonzero
 * number).  When on, nova_kv_encode, nova_kv_decode_attn and
 * nova_kv_append_decode_attn (and its allocation-free variant) wait for their
 * stream, copy seq_lens / start_pos / the block table to the host and run
 * nova_kv_check_metadata (with num_blocks as given here, <= 0: unknown)
 * before launching; a failing check launches nothing.  This synchronizes,
 * so it is for debugging and not for graph capture.
 */
void nova_kv_set_debug(int32_t on, int32_t num_blocks);

/* Static description of a status code. */
const char *nova_kv_status_string(nova_kv_status s);

/* Detail of the last failing call on this thread ("" if none). */
const char *nova_kv_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* NOVA_KV_H */
