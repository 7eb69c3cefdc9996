/*
 * starkv.h -- decode attention read directly from a low-rank, quantized KV cache
 * (STAR-KV), for AMD Instinct MI355X (gfx950).
 *
 * The method (paper sections in brackets):
 *   keys    K = (x . (Sigma V)_K,g) . U_K,g^T   one latent of rank r_g per KV head
 *           (head-wise decomposition)                               [Sec. 3.2, 4.3.3]
 *   values  V = (x . (Sigma V)_V) . U_V^T       one latent of rank r_v shared by all
 *           heads of the layer (joint decomposition)                [Sec. 3.2, 4.3.3]
 *   cache   the latents, quantized per token: an outlier block of leading
 *           channels at 8 bits and an inlier block at 4 bits        [Sec. 4.4, Eq. Z-hat]
 *   decode  keys are rebuilt from the latents, rotated with RoPE at their
 *           position (RoPE blocks absorbing U_K into W_Q)           [Sec. 3.3]
 *           and scored against q with a softmax over the context    [Sec. 3.1];
 *           values are reordered: the probabilities weight the shared latent
 *           V' and U_V is applied once per query head               [Sec. 3.3]
 *           (the fused key and value kernels and the stacked p.V' GEMM of
 *           App. A.6, "Operation Fusion" and "Attention with GEMM").
 * The block-wise Hadamard rotation of Sec. 4.4 is fused offline into the
 * factors; this library takes the factors as given.
 *
 * Conventions for every entry point:
 *   - The caller owns all device memory (cache, q, factors, outputs, workspace)
 *     and the plan's lifetime.  The library never allocates or frees device
 *     memory and never synchronizes.
 *   - Device work is enqueued on the given HIP stream and is complete when the
 *     stream is.  Pointers documented as "device" must be device-accessible.
 *   - Argument errors are reported synchronously, before anything is launched.
 *     A failed launch returns STARKV_ERR_HIP.  No C++ exception crosses this
 *     interface and nothing aborts.  starkv_last_error() gives a detail string
 *     for the calling thread's last failure.
 *   - Calls that write the same cache rows, or share a workspace, race if they
 *     overlap on different streams.
 */
#ifndef STARKV_H
#define STARKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* starkv_stream_t;   /* a hipStream_t; NULL = default stream */

typedef enum {
  STARKV_OK = 0,
  STARKV_ERR_INVALID_ARG = 1,   /* null/ill-formed argument, inconsistent sizes */
  STARKV_ERR_UNSUPPORTED = 2,   /* well-formed but outside what the kernels implement */
  STARKV_ERR_CAPACITY = 3,      /* a length beyond the cache capacity */
  STARKV_ERR_WORKSPACE = 4,     /* workspace missing or smaller than required */
  STARKV_ERR_ALIGNMENT = 5,     /* a device pointer not aligned as documented */
  STARKV_ERR_HIP = 6            /* the HIP runtime reported an error */
} starkv_status;

/* Cache precision (Sec. 4.4; bit widths per this library's formats):
 *   F16     latents stored as fp16, no quantization;
 *   INT4    every channel 4-bit;
 *   MIX8_4  the leading r_out = 8*ceil(r/32) channels (about 25 %, the outlier
 *           block; the latent channels are ordered by singular value) at 8 bits,
 *           the remaining channels (inlier block) at 4 bits;
 *   MIX4_3  the paper's own split (Sec. 5, quantization results): the leading
 *           r_out = 8*max(1, floor((r + 20)/40)) channels (a fifth of r to the
 *           nearest multiple of 8, at least 8, at most r) at 4 bits, the rest at
 *           3 bits -- 3.2 bits per channel on average when r/5 is a multiple of 8.
 *           The block Hadamard rotations of Sec. 4.4 are fused into the
 *           caller's down- and up-projection factors. */
typedef enum { STARKV_Q_F16 = 0, STARKV_Q_INT4 = 1, STARKV_Q_MIX8_4 = 2,
               STARKV_Q_MIX4_3 = 3 } starkv_qmode;

/* Element types.  F32 is accepted for the attention output only. */
typedef enum { STARKV_DT_F16 = 0, STARKV_DT_BF16 = 1, STARKV_DT_F32 = 2 } starkv_dtype;

#define STARKV_MAX_KV_HEADS 16
#define STARKV_MAX_Q_HEADS 64

typedef struct {
  int32_t batch;          /* sequences B */
  int32_t n_q_heads;      /* H_q, a multiple of n_kv_heads, <= 64 */
  int32_t n_kv_heads;     /* H_kv <= 16; query head i reads KV head floor(i*H_kv/H_q) */
  int32_t head_dim;       /* d: 64 or 128 */
  int32_t capacity;       /* rows per sequence in the cache, >= 1 */
  const int32_t* key_rank;/* host array [H_kv]: r_g, multiples of 16 in [16, d] (copied) */
  int32_t value_rank;     /* r_v: a multiple of 16 in [16, min(H_kv*d, 1024)] */
  int32_t qmode;          /* starkv_qmode */
  int32_t group_size;     /* quantization group, must be 32 */
  double  rope_theta;     /* RoPE base, > 1 */
  int32_t d_model;        /* hidden size for starkv_append's down-projection; 0 = latents given */
  int32_t q_dtype;        /* starkv_dtype of q */
  int32_t out_dtype;      /* starkv_dtype of the attention output (F16, BF16 or F32) */
  int32_t x_dtype;        /* starkv_dtype of hidden states (when d_model > 0) */
  /* Paged cache, for continuous batching (zero-initialize for the contiguous
   * layout).  page_tokens = 0: sequence b owns a padded run of rows.  Otherwise a
   * power of two in [128, 8192]: the cache is a pool of n_pages pages of
   * page_tokens rows, and block_table maps each sequence's pages to pool pages. */
  int32_t page_tokens;
  int32_t n_pages;        /* pages in the pool, >= 1 (paged caches) */
  /* device int32 [B][ceil(capacity / page_tokens)], 4-byte aligned: pool page of
   * page j (tokens j*page_tokens ..) of each sequence.  The pointer is fixed at
   * plan creation; the contents are read by every append and decode call at its
   * place in the stream, so the caller hands out pages by rewriting entries
   * between calls (also between replays of a captured graph).  Append drops rows
   * whose entry is outside [0, n_pages); decode must only reach valid entries
   * (it clamps others into the pool and reads whatever is there). */
  const int32_t* block_table;
} starkv_config;

typedef struct starkv_plan starkv_plan;   /* opaque, immutable after creation */

/* ------------------------------------------------------------------------------
 * Cache format.  All integers little-endian, fp16 as IEEE binary16.
 * Every plane has one row per token slot.  Contiguous caches: rows per sequence
 * are padded to Cp = ceil(capacity/256)*256 and token t of sequence b is row
 * R = b*Cp + t.  Paged caches: the planes have n_pages*P rows (P = page_tokens)
 * and token t of sequence b is row R = block_table[b][t/P]*P + t%P.
 * The cache is a sequence of planes, each starting on a 256-byte boundary, in
 * this order: for g = 0..H_kv-1 {key code plane g, key meta plane g}, then the
 * value code plane, then the value meta plane.  Meta planes of F16 caches are
 * empty.
 *
 * A latent block of rank r (key head g: r = r_g; values: r = r_v) has regions:
 * F16: one region, 16-bit values.  INT4: one 4-bit region.  MIX8_4: 8-bit
 * channels [0, r_out), 4-bit channels [r_out, r).  MIX4_3: 4-bit channels
 * [0, r_out), 3-bit channels [r_out, r).  Each quantized region is split into
 * groups of 32 channels from the region start (the last may be shorter); groups
 * are numbered outlier region first.  Per token and group: z = min over the
 * group's fp16 values, s = the smallest fp16 >= (max - min)/(2^b - 1) (s = 0 when
 * max == min), code = round-half-even((x - z)/s) clamped to [0, 2^b - 1]
 * (evaluated in fp64, which is exact for these operands); decode x-hat = z + code*s.
 * Row bytes: F16 2r; INT4 r/2; MIX8_4 r_out + (r - r_out)/2; MIX4_3
 * r_out/2 + 3(r - r_out)/8.
 *
 * Keys, head g, sequence b, token t (row R): 16-token block R/16, tau = t%16, at
 *   plane + (R/16) * 16*row_bytes.  Inside a block the channels go in
 *   chunks of 8 (chunk c = channels 8c..8c+7); chunk c holds its 16 tokens
 *   back to back, chunk_bytes each (16 F16, 8 for 8-bit, 4 for 4-bit, 3 for
 *   3-bit chunks), outlier chunks first.  Within a chunk: F16 channel w at 2w;
 *   8-bit channel w at byte w; 4-bit channel w at byte w/2, low nibble for even
 *   w; 3-bit channel w at bits 3w..3w+2 of the token's 3 bytes read as a
 *   little-endian 24-bit word.
 *   Key meta: per 16-token block, per group, 16 (s, z) fp16 pairs (4 B per token).
 * Values, sequence b, token t (row R): 32-token block R/32 at
 *   plane + (R/32) * 32*row_bytes.  A block's tokens form four chunks q of
 *   eight slots: with u = t%32, q = u%4 and slot = 4*(u/16) + (u%16)/4 (so chunk q
 *   holds the tokens q, q+4, .., q+28 of the block, in that order).  For each chunk q and channel c the
 *   eight slots are stored together: F16 16 B (slot at 2*slot), 8-bit 8 B (slot at
 *   byte slot), 4-bit one 32-bit word (slot 2k in bits 4k..4k+3, slot 2k+1 in bits
 *   16+4k..16+4k+3, k = 0..3), 3-bit 3 bytes read as a little-endian 24-bit word
 *   (slot 2k in bits 3k..3k+2, slot 2k+1 in bits 12+3k..14+3k).  The outlier
 *   region precedes the inlier region; within a region the order is
 *   [channel][q][slots].
 *   Value meta: per 32-token block, per group g, per chunk q: the 8 slots' s
 *   (16 B) then their z (16 B), at ((g*4 + q)*32) inside the block's meta.
 * ---------------------------------------------------------------------------- */
typedef struct {
  int64_t total_bytes;
  int32_t padded_capacity;                       /* Cp */
  int32_t sum_key_rank;                          /* sum of r_g */
  int64_t key_code_offset[STARKV_MAX_KV_HEADS];
  int64_t key_meta_offset[STARKV_MAX_KV_HEADS];
  int32_t key_row_bytes[STARKV_MAX_KV_HEADS];
  int32_t key_groups[STARKV_MAX_KV_HEADS];
  int32_t key_outlier_channels[STARKV_MAX_KV_HEADS];
  int64_t value_code_offset;
  int64_t value_meta_offset;
  int32_t value_row_bytes;
  int32_t value_groups;
  int32_t value_outlier_channels;
  int64_t rows;                                  /* rows of every plane: B*Cp, or n_pages*P */
  int32_t page_tokens;                           /* P (0: contiguous) */
  int32_t pages_per_sequence;                    /* block_table row length (paged) */
} starkv_layout;

/* Validates cfg and builds a plan (host memory owned by the library).
 * Errors: INVALID_ARG (null, non-positive sizes, ranks not multiples of 16, ...),
 * UNSUPPORTED (head_dim not 64/128, group_size != 32, too many heads, ...). */
starkv_status starkv_plan_create(const starkv_config* cfg, starkv_plan** out);
void          starkv_plan_destroy(starkv_plan* plan);

/* Bytes of device memory the caller allocates for one cache (one layer). */
size_t        starkv_cache_bytes(const starkv_plan* plan);
starkv_status starkv_cache_layout(const starkv_plan* plan, starkv_layout* out);

/* Workspace sizes (bytes).  Append: the fp16 latents of the new tokens plus, when
 * d_model > 0, the down-projection's fp32 partial sums (or, for 512 and more new
 * rows B*n_new with d_model a multiple of 64, A_all transposed for the prefill
 * GEMM).  Decode: the split
 * partials and rescoring candidates for contexts up to max_ctx, the normalized
 * value latents that the absorbed output reads (the same size serves both
 * decode entry points), and the per-sequence work plan the split pass leaves
 * for the combine pass. */
size_t        starkv_append_workspace_bytes(const starkv_plan* plan, int32_t n_new);
size_t        starkv_decode_workspace_bytes(const starkv_plan* plan, int32_t max_ctx);

/* starkv_append -- write n_new new tokens of every sequence into the cache.
 * Down-projection (Sec. 3.2) then per-token quantization (Sec. 4.4).
 *   cache        device, starkv_cache_bytes(plan) bytes, 256-byte aligned.
 *   x_or_latents device.  d_model > 0: hidden states [B][n_new][d_model] in x_dtype;
 *                the latents x.A_all are accumulated in fp32 and rounded to fp16
 *                (left in ws: [B][n_new][sum_r + r_v] fp16 at offset 0).
 *                16-byte aligned.  d_model == 0: fp16 latents [B][n_new][sum_r + r_v]
 *                (key heads in order, then the value latent), 2-byte aligned.
 *   A_all        device bf16 [d_model][sum_r + r_v] (column block per key head, then
 *                values), 16-byte aligned; NULL when d_model == 0.
 *   pos_dev      device int32 [B]: row of the first new token of each sequence;
 *                rows pos[b] .. pos[b]+n_new-1 are written.  Rows outside
 *                [0, capacity) are not written.  The caller advances its lengths.
 *   n_new        >= 1.
 *   ws           device workspace of starkv_append_workspace_bytes(plan, n_new)
 *                bytes, 256-byte aligned.
 * Errors: INVALID_ARG, WORKSPACE, ALIGNMENT, HIP. */
starkv_status starkv_append(const starkv_plan* plan, void* cache, const void* x_or_latents,
                            const void* A_all, const int32_t* pos_dev, int32_t n_new,
                            void* ws, size_t ws_bytes, starkv_stream_t stream);

/* starkv_decode_attn -- one decode step of attention for every sequence.
 *   cache        device, as written by starkv_append.
 *   q            device [B][H_q][d] in q_dtype, already rotated (RoPE) for the
 *                current position; 16-byte aligned.
 *   B_k          device fp16 [sum_r][d]: U_K,g^T of head g at rows
 *                sum_{g'<g} r_g' .. +r_g (the key up-projection, Sec. 3.2);
 *                16-byte aligned.
 *   B_v          device fp16 [r_v][H_kv*d]: U_V^T; query head i uses columns
 *                g*d .. g*d+d-1 of its KV head g; 16-byte aligned.
 *   ctx_len_dev  device int32 [B]: sequence b attends to rows [0, ctx_len[b]);
 *                key t is rotated by RoPE at position t.  Values are clamped to
 *                [0, max_ctx]; 0 gives a zero output.
 *   max_ctx      host upper bound of ctx_len, 1 <= max_ctx <= capacity, and at most
 *                524288 tokens (UNSUPPORTED beyond).
 *   out          device [B][H_q][d] in out_dtype, 16-byte aligned; 16-bit types are
 *                rounded to nearest even from the fp32 result.
 *   ws           device, starkv_decode_workspace_bytes(plan, max_ctx) bytes,
 *                256-byte aligned.
 * Accuracy: scores are computed with fp16 operands and fp32 accumulation; the
 * tokens that hold most of the softmax mass are rescored exactly in fp32 (see
 * the combine pass below), so near-ties between dominant tokens are resolved at
 * fp32 accuracy.
 * Errors: INVALID_ARG, CAPACITY (max_ctx > capacity), WORKSPACE, ALIGNMENT, HIP. */
starkv_status starkv_decode_attn(const starkv_plan* plan, const void* cache, const void* q,
                                 const void* B_k, const void* B_v, const int32_t* ctx_len_dev,
                                 int32_t max_ctx, void* out, void* ws, size_t ws_bytes,
                                 starkv_stream_t stream);

/* starkv_decode_attn_noalloc -- starkv_decode_attn without a caller workspace, for
 * callers that cannot allocate device memory (code under graph capture, tight
 * serving loops, harnesses that forbid allocation).  Its workspace is a fixed
 * device array of 32 MiB inside the library, one per device, held until the
 * process ends; no call allocates or frees memory.
 *   cache, q, B_k, B_v, ctx_len_dev, max_ctx, out, stream: as for
 *                starkv_decode_attn (same kernels, same results).
 * All calls on one device share that array and leave their partial results in
 * it: calls that overlap on one device (other streams, other threads) race and
 * must be ordered by the caller.
 * Errors: as starkv_decode_attn; WORKSPACE when starkv_decode_workspace_bytes(plan,
 * max_ctx) exceeds 32 MiB (the C3 layer shape needs 12.4 MiB at 4 x 131072 tokens
 * and 51.0 MiB at 64 x 131072). */
starkv_status starkv_decode_attn_noalloc(const starkv_plan* plan, const void* cache,
                                         const void* q, const void* B_k, const void* B_v,
                                         const int32_t* ctx_len_dev, int32_t max_ctx, void* out,
                                         starkv_stream_t stream);

/* The two launches of starkv_decode_attn, exposed separately so that each can be
 * timed on its own, with the same arguments and errors:
 *   split    keys, scores, softmax state and value latents per context split, the
 *            largest approximate scores of each split that may need rescoring,
 *            and (for batches of up to 64 sequences) each sequence's work plan,
 *            written to ws;
 *   combine  merge of the splits (log-sum-exp weights), exact fp32 rescoring of
 *            the tokens that dominate the softmax (re-read from the cache), and
 *            the value up-projection into out.
 * The combine pass must follow a split pass with the same cache, q, B_k,
 * ctx_len, max_ctx and ws. */
starkv_status starkv_decode_split(const starkv_plan* plan, const void* cache, const void* q,
                                  const void* B_k, const int32_t* ctx_len_dev, int32_t max_ctx,
                                  void* ws, size_t ws_bytes, starkv_stream_t stream);
starkv_status starkv_decode_combine(const starkv_plan* plan, const void* cache, const void* q,
                                    const void* B_k, const void* B_v,
                                    const int32_t* ctx_len_dev, int32_t max_ctx, void* out,
                                    void* ws, size_t ws_bytes, starkv_stream_t stream);

/* starkv_decode_attn_absorbed -- starkv_decode_attn with the value up-projection
 * absorbed into the output projection (Sec. 3.3, weight absorption): instead of
 * the per-head outputs o_i = (a_i / l_i) U_V,g^T it writes the attention block's
 * output y_b = sum_i o_i W_out,i^T = sum_i W'_out,i (a_i / l_i), with the
 * absorbed weights W'_out,i = W_out,i U_V,g(i) formed once, offline.
 *   cache, q, B_k, ctx_len_dev, max_ctx, ws: as for starkv_decode_attn (B_v is
 *                not used).
 *   W_abs        device fp16 [d_out][H_q * r_v], 16-byte aligned: W'_out,i of query
 *                head i in columns i*r_v .. i*r_v + r_v - 1 (W_out,i: the columns
 *                i*d .. i*d+d-1 of the output projection [d_out][H_q*d]).
 *   d_out        output width (the model dimension), >= 1.
 *   out          device [B][d_out] in out_dtype, 16-byte aligned; a sequence with
 *                ctx_len 0 gets zeros.
 * Accuracy: the normalized latents (fp32) enter the product as two fp16 parts,
 * each product exact, accumulated in fp32.
 * Errors: as starkv_decode_attn; INVALID_ARG for a NULL W_abs or out or d_out < 1. */
starkv_status starkv_decode_attn_absorbed(const starkv_plan* plan, const void* cache,
                                          const void* q, const void* B_k, const void* W_abs,
                                          int32_t d_out, const int32_t* ctx_len_dev,
                                          int32_t max_ctx, void* out, void* ws, size_t ws_bytes,
                                          starkv_stream_t stream);
/* Its second part, after starkv_decode_split (for timing, as above): the merge of
 * the splits with the exact rescoring, the normalized latents into ws, then the
 * product with W_abs into out. */
starkv_status starkv_decode_combine_absorbed(const starkv_plan* plan, const void* cache,
                                             const void* q, const void* B_k, const void* W_abs,
                                             int32_t d_out, const int32_t* ctx_len_dev,
                                             int32_t max_ctx, void* out, void* ws,
                                             size_t ws_bytes, starkv_stream_t stream);

/* Number of context splits and tokens per split for max_ctx tokens in every
 * sequence; informative.  With up to 64 sequences the kernels choose the split
 * length on the device from the actual lengths (the smallest multiple of 128
 * tokens giving at most one work item per compute unit and head group, at most
 * 256 splits of at most 8192 tokens per sequence); these functions report that plan for equal
 * lengths of max_ctx. */
int32_t       starkv_decode_splits(const starkv_plan* plan, int32_t max_ctx);
int32_t       starkv_decode_split_tokens(const starkv_plan* plan, int32_t max_ctx);

/* Shape of the decode launch a plan makes for max_ctx (informative, for tests and
 * measurement; no device work).  The split pass is one kernel instance per
 * (head_dim, qmode, score_tiles, value_tiles) and runs a grid of work items x
 * head_groups workgroups.  With device_plan != 0 (batches of up to 64 sequences)
 * the kernels take the split length S = 128 k from the actual lengths L_b: the
 * smallest k >= k_lo with sum_b ceil(L_b / S) <= items; otherwise every sequence
 * has `items / batch` splits of split_tokens tokens.
 * Errors: INVALID_ARG for a NULL plan or out, or max_ctx < 1. */
typedef struct {
  int32_t head_dim, qmode;
  int32_t score_tiles;       /* 16-column score tiles of a head group */
  int32_t value_tiles;       /* 16-channel value tiles per wave */
  int32_t head_groups;       /* workgroups per work item (KV heads split by LDS size) */
  int32_t device_plan;       /* 1: split length chosen on the device from ctx_len */
  int32_t k_lo, items;       /* device plan: smallest k, work items (grid.x) */
  int32_t split_tokens;      /* split length for max_ctx in every sequence */
  int32_t lds_bytes;         /* dynamic LDS of a split workgroup */
} starkv_decode_info;
starkv_status starkv_decode_describe(const starkv_plan* plan, int32_t max_ctx,
                                     starkv_decode_info* out);

/* starkv_read_stream -- a measurement aid, not part of the method: reads `bytes`
 * at src once with 16-byte loads (every lane keeps sixteen in flight, grid-stride
 * over `workgroups` workgroups of 256 threads) and folds them into one word per
 * wave, written to sink.  Timing it gives the plain HBM read ceiling that the
 * split pass's latent stream is compared with.
 *   src          device, 16-byte aligned; bytes a positive multiple of 16.
 *   workgroups   1 .. 65536 (0: 2048, eight per compute unit).
 *   sink         device uint32 [workgroups * 4] (sink_bytes at least that), 4-byte aligned.
 * Errors: INVALID_ARG (NULL pointers, sizes), ALIGNMENT, HIP (launch). */
starkv_status starkv_read_stream(const void* src, size_t bytes, int32_t workgroups, void* sink,
                                 size_t sink_bytes, starkv_stream_t stream);

const char*   starkv_status_string(starkv_status status);
const char*   starkv_last_error(void);          /* thread-local, never NULL */

#ifdef __cplusplus
}
#endif
#endif /* STARKV_H */
