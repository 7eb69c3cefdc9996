/*
 * STAR-KV decode-path oracle: plain, slow, fp64 CPU reference.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this code; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no source with the HIP path: its own
 * config struct, its own fp16 conversions, its own layout addressing.
 *
 * What it computes (paper sections cited per function in oracle.c):
 *   - down-projection of hidden states into latents (Sec. 3.2),
 *   - per-token group quantization of the latents into an outlier and an
 *     inlier region (Sec. 4.4, Eq. for Z-hat): 8/4 bits, or the paper's own
 *     4/3 bits with about 20 % outliers (Sec. 5, quantization results),
 *   - the cache byte layout (this library's format, documented in the
 *     public header of the product library; re-derived here independently),
 *   - decode attention read from that cache: dequantize, reconstruct keys
 *     per KV head (head-wise decomposition, Sec. 4.3.3), RoPE (Sec. 3.3),
 *     softmax attention (Sec. 3.1), value latents accumulated with the
 *     shared value latent and up-projected once per query head (the
 *     reordering of Sec. 3.3 with joint decomposition for values, Sec. 4.3.3),
 *   - dense attention from explicit K and V (Sec. 3.1), used only by tests.
 */
#ifndef STARKV_ORACLE_H
#define STARKV_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_Q_F16 = 0, ORC_Q_INT4 = 1, ORC_Q_MIX8_4 = 2, ORC_Q_MIX4_3 = 3 };

typedef struct {
  int32_t batch, n_q_heads, n_kv_heads, head_dim, capacity;
  int32_t key_rank[64];   /* per KV head */
  int32_t value_rank;     /* one value latent shared by all heads */
  int32_t qmode;
  double  rope_theta;
  int32_t d_model;
  /* paged layout (page_tokens > 0): the cache is a pool of n_pages pages of
   * page_tokens rows; token t of sequence b lives in row
   * table[b][t / page_tokens] * page_tokens + t % page_tokens, with table
   * [batch][ceil(capacity / page_tokens)] (host memory).  page_tokens == 0:
   * sequence b owns rows b * padded capacity + t. */
  int32_t page_tokens, n_pages;
  const int32_t* table;
} orc_cfg;

/* ---- fp16 / bf16 (own implementations of the IEEE formats) ---- */
double   orc_f16_to_double(uint16_t h);
uint16_t orc_double_to_f16(double x);          /* round to nearest, ties to even */
uint16_t orc_f16_ceil(double q);               /* smallest fp16 >= q, q >= 0 */
double   orc_bf16_to_double(uint16_t b);

/* ---- quantizer: one latent block of rank r for one token ----
 * x: r fp16 values.  codes: r entries (0 .. 2^bits - 1; raw fp16 bits for F16
 * are not produced here).  s, z: one fp16 pair per group, outlier groups first.
 * Returns the number of groups. */
int orc_n_groups(int qmode, int r);
int orc_outlier_channels(int qmode, int r);
int orc_quantize_block(int qmode, int r, const uint16_t* x,
                       uint8_t* codes, uint16_t* s, uint16_t* z);
/* group index and bit width of channel c in a block of rank r */
int orc_channel_group(int qmode, int r, int c, int* bits);

/* ---- cache layout ---- */
int64_t orc_cache_bytes(const orc_cfg* cfg);
/* byte offsets of the planes (for cross-checking the library's layout query) */
int64_t orc_plane_offset(const orc_cfg* cfg, int which, int head);  /* which: 0 K codes, 1 K meta, 2 V codes, 3 V meta */

/* append n_new tokens of latents [B][n_new][sum_r + r_v] fp16 at rows pos[b]+j
 * (rows outside the cache are dropped).  Returns 0, or -1 (nothing written) for a
 * batch above 1024 or a negative n_new. */
int orc_append(const orc_cfg* cfg, uint8_t* cache, const uint16_t* latents,
               const int32_t* pos, int n_new);

/* down-projection: latents = round_fp16( x[B*n_new][d_model] . A[d_model][sum_r+r_v] );
 * x_is_bf16 selects bf16 (1) or fp16 (0) hidden states; A is bf16. z64 (optional)
 * receives the unrounded fp64 products. */
int orc_downproj(const orc_cfg* cfg, const uint16_t* x, int x_is_bf16,
                 const uint16_t* A, int n_tok, uint16_t* latents, double* z64);

/* dequantized latents of one token read back from the cache:
 * khat [sum_r] (heads in order), vhat [r_v] */
int orc_read_token(const orc_cfg* cfg, const uint8_t* cache, int b, int t,
                   double* khat, double* vhat);

/* reconstructed key of KV head g at cache row t, before (rope=0) or after RoPE */
int orc_reconstruct_key(const orc_cfg* cfg, const uint8_t* cache,
                        const uint16_t* Bk, int b, int g, int t, int rope, double* k);

/* rotate-half RoPE of a d-vector at position t (in place) */
void orc_rope(double* v, int d, double t, double theta);

/* decode attention.  q [B][H_q][d] (bf16 if q_is_bf16 else fp16), Bk [sum_r][d] fp16,
 * Bv [r_v][H_kv*d] fp16, ctx_len [B].  out [B][H_q][d] fp64.  If sel != NULL only the
 * n_sel (b, query head) pairs sel[2k], sel[2k+1] are computed (others untouched).
 * n_threads <= 0 means one thread per hardware core. Returns threads used, or -1
 * (nothing computed) when a ctx_len is negative or above the capacity, or a
 * selected pair is out of range. */
int orc_decode_attn(const orc_cfg* cfg, const uint8_t* cache, const uint16_t* q,
                    int q_is_bf16, const uint16_t* Bk, const uint16_t* Bv,
                    const int32_t* ctx_len, const int32_t* sel, int n_sel,
                    double* out, int n_threads);

/* the same pass up to the normalized value latent: lat [B][H_q][r_v] fp64 gets
 * a_i / l_i (zero for ctx_len == 0) for the selected (b, head) pairs; errors as
 * for orc_decode_attn. */
int orc_decode_latent(const orc_cfg* cfg, const uint8_t* cache, const uint16_t* q,
                      int q_is_bf16, const uint16_t* Bk, const int32_t* ctx_len,
                      const int32_t* sel, int n_sel, double* lat, int n_threads);

/* dense attention for one query head from explicit pre-RoPE keys and values:
 * q[d], K[L][d], V[L][d] (fp64) -> out[d]; RoPE applied to K at positions 0..L-1 */
void orc_dense_attn(int d, int L, const double* q, const double* K,
                    const double* V, double theta, double* out);

#ifdef __cplusplus
}
#endif
#endif
