/*
 * STAR-KV decode-path oracle (fp64, plain loops).  TEST INFRASTRUCTURE ONLY:
 * used by the tests, the smoke check and the benchmark's CPU-baseline leg,
 * never by the product path.  See oracle.h for the list of what it computes.
 *
 * Every arithmetic step is written the slow, direct way: fp64 throughout,
 * no blocking, no fusion, one loop per formula.
 */
#include "oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

/* ------------------------------------------------------------------------ */
/* fp16 and bf16, from the IEEE 754 binary16 definition and bf16 = top half  */
/* of binary32.                                                             */
/* ------------------------------------------------------------------------ */

double orc_f16_to_double(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 31;
  int m = h & 1023;
  double v;
  if (e == 0) {
    v = ldexp((double)m, -24);                 /* subnormal: m * 2^-24 */
  } else if (e == 31) {
    v = m ? NAN : INFINITY;
  } else {
    v = ldexp((double)(1024 + m), e - 25);     /* (1 + m/1024) * 2^(e-15) */
  }
  return sign ? -v : v;
}

uint16_t orc_double_to_f16(double x) {
  uint16_t sign = signbit(x) ? 0x8000 : 0;
  double a = fabs(x);
  if (isnan(x)) return 0x7E00;
  if (a >= 65520.0) return sign | 0x7C00;      /* rounds to infinity */
  if (a < ldexp(1.0, -14)) {
    /* subnormal range: value = m * 2^-24, m rounded to nearest even */
    double m = nearbyint(ldexp(a, 24));
    return sign | (uint16_t)m;                 /* m == 1024 is the smallest normal */
  }
  int E;
  frexp(a, &E);                                /* a = f * 2^E, f in [0.5, 1) */
  int e = E - 1;                               /* a in [2^e, 2^(e+1)) */
  double m = nearbyint(ldexp(a, 10 - e));      /* in [1024, 2048] */
  if (m == 2048.0) { m = 1024.0; e += 1; }
  if (e > 15) return sign | 0x7C00;
  return sign | (uint16_t)(((e + 15) << 10) | ((int)m - 1024));
}

uint16_t orc_f16_ceil(double q) {
  /* Positive fp16 bit patterns 0x0000..0x7C00 are ordered like their values,
   * so the smallest fp16 >= q is found by bisection over the patterns. */
  if (!(q > 0.0)) return 0;
  uint16_t lo = 0, hi = 0x7C00;                /* value(hi) = +inf >= q */
  while (lo < hi) {
    uint16_t mid = (uint16_t)((lo + hi) / 2);
    if (orc_f16_to_double(mid) >= q) hi = mid; else lo = (uint16_t)(mid + 1);
  }
  return lo;
}

double orc_bf16_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* ------------------------------------------------------------------------ */
/* Quantizer (Sec. 4.4): per token, the latent block is split into an        */
/* outlier region (leading channels, largest singular values, b_out bits)    */
/* and an inlier region (b_in bits); each region is quantized per token in   */
/* groups of 32 channels with an asymmetric min/max scale and zero point.    */
/* ------------------------------------------------------------------------ */

#define GROUP 32

/* Bit widths of the two regions of a latent block: the outlier region takes
 * the leading channels (largest singular values), the inlier region the rest.
 * MIX8_4: 8 / 4 bits.  MIX4_3: the paper's own split, 4-bit outliers and
 * 3-bit inliers.  INT4: a single 4-bit region. */
static int hi_bits(int qmode) { return qmode == ORC_Q_MIX8_4 ? 8 : 4; }
static int lo_bits(int qmode) { return qmode == ORC_Q_MIX4_3 ? 3 : 4; }

int orc_outlier_channels(int qmode, int r) {
  if (qmode == ORC_Q_MIX8_4) return 8 * ((r + 31) / 32);   /* 25 % of r, rounded up to 8 */
  if (qmode == ORC_Q_MIX4_3) {
    /* 20 % of r to the nearest multiple of 8 (halves up), at least 8 */
    int ro = 8 * ((r + 20) / 40);
    if (ro < 8) ro = 8;
    return ro < r ? ro : r;
  }
  return 0;
}

int orc_n_groups(int qmode, int r) {
  if (qmode == ORC_Q_F16) return 0;
  int ro = orc_outlier_channels(qmode, r);
  return (ro + GROUP - 1) / GROUP + (r - ro + GROUP - 1) / GROUP;
}

int orc_channel_group(int qmode, int r, int c, int* bits) {
  if (qmode == ORC_Q_F16) { *bits = 16; return -1; }
  int ro = orc_outlier_channels(qmode, r);
  if (c < ro) { *bits = hi_bits(qmode); return c / GROUP; }
  *bits = lo_bits(qmode);
  return (ro + GROUP - 1) / GROUP + (c - ro) / GROUP;
}

int orc_quantize_block(int qmode, int r, const uint16_t* x,
                       uint8_t* codes, uint16_t* s, uint16_t* z) {
  int ng = orc_n_groups(qmode, r);
  for (int gi = 0; gi < ng; ++gi) {
    /* members of group gi */
    double lo = INFINITY, hi = -INFINITY;
    int bits = 0;
    for (int c = 0; c < r; ++c) {
      int b;
      if (orc_channel_group(qmode, r, c, &b) != gi) continue;
      bits = b;
      double v = orc_f16_to_double(x[c]);
      if (v < lo) lo = v;
      if (v > hi) hi = v;
    }
    double levels = (double)((1 << bits) - 1);
    uint16_t s16 = 0;                          /* hi == lo: scale 0, all codes 0 */
    if (hi > lo) s16 = orc_f16_ceil((hi - lo) / levels);
    double sv = orc_f16_to_double(s16);
    s[gi] = s16;
    z[gi] = orc_double_to_f16(lo);             /* lo is an fp16 value: exact */
    for (int c = 0; c < r; ++c) {
      int b;
      if (orc_channel_group(qmode, r, c, &b) != gi) continue;
      double code = 0.0;
      if (sv > 0.0) {
        code = nearbyint((orc_f16_to_double(x[c]) - lo) / sv);
        if (code < 0.0) code = 0.0;
        if (code > levels) code = levels;
      }
      codes[c] = (uint8_t)code;
    }
  }
  return ng;
}

/* ------------------------------------------------------------------------ */
/* Cache layout.  Capacity is padded to a multiple of 256 rows.  Planes, in  */
/* order, each starting on a 256-byte boundary: for every KV head g its key  */
/* code plane and key meta plane, then the value code plane and value meta   */
/* plane.  Keys are tiled in 16-token blocks, values in 32-token blocks.     */
/* A plane has one row per token slot: per sequence a padded run of rows,  */
/* or, paged, a pool of pages that a block table hands out to sequences.    */
/* ------------------------------------------------------------------------ */

static int64_t pad_cap(const orc_cfg* c) { return ((int64_t)c->capacity + 255) / 256 * 256; }
static int64_t align256(int64_t x) { return (x + 255) / 256 * 256; }

/* Rows of every plane: one padded run per sequence, or the page pool. */
static int64_t plane_rows(const orc_cfg* c) {
  return c->page_tokens > 0 ? (int64_t)c->n_pages * c->page_tokens
                            : (int64_t)c->batch * pad_cap(c);
}

/* Row of token t of sequence b, or -1 when its page is not a pool page. */
static int64_t row_of(const orc_cfg* c, int b, int t) {
  if (c->page_tokens <= 0) return (int64_t)b * pad_cap(c) + t;
  int per_seq = (c->capacity + c->page_tokens - 1) / c->page_tokens;
  int32_t pg = c->table[(int64_t)b * per_seq + t / c->page_tokens];
  if (pg < 0 || pg >= c->n_pages) return -1;
  return (int64_t)pg * c->page_tokens + t % c->page_tokens;
}

static int row_bytes(int qmode, int r) {
  if (qmode == ORC_Q_F16) return 2 * r;
  int ro = orc_outlier_channels(qmode, r);
  return ro * hi_bits(qmode) / 8 + (r - ro) * lo_bits(qmode) / 8;
}

int64_t orc_plane_offset(const orc_cfg* cfg, int which, int head) {
  int64_t rows = plane_rows(cfg);
  int64_t off = 0;
  for (int g = 0; g < cfg->n_kv_heads; ++g) {
    int r = cfg->key_rank[g];
    if (which == 0 && head == g) return off;
    off = align256(off + rows * row_bytes(cfg->qmode, r));
    if (which == 1 && head == g) return off;
    off = align256(off + rows * 4 * orc_n_groups(cfg->qmode, r));
  }
  if (which == 2) return off;
  off = align256(off + rows * row_bytes(cfg->qmode, cfg->value_rank));
  if (which == 3) return off;
  off = align256(off + rows * 4 * orc_n_groups(cfg->qmode, cfg->value_rank));
  return off;                                  /* which == 4: total */
}

int64_t orc_cache_bytes(const orc_cfg* cfg) { return orc_plane_offset(cfg, 4, 0); }

/* Key code of channel c of head g at token t.  Returns the byte offset of the
 * code's container and, in *bit, the code's first bit in it (containers: one
 * byte for 8-bit and 4-bit codes, two for fp16, three for 3-bit codes read as
 * a little-endian 24-bit word).  Within a 16-token block the channels are
 * taken in chunks of 8, outlier chunks first; each chunk stores its 16 tokens
 * contiguously, a token's 8 codes in b bytes (b = bits per code):
 *   8-bit: channel w in byte w;  4-bit: channel w in byte w/2, low nibble for
 *   even w;  3-bit: channel w at bits 3w..3w+2 of the token's 24-bit word. */
static int64_t key_code_at(const orc_cfg* cfg, int g, int b, int t, int c, int* bit) {
  int r = cfg->key_rank[g];
  int rb = row_bytes(cfg->qmode, r);
  int64_t base = orc_plane_offset(cfg, 0, g) + (row_of(cfg, b, t) / 16) * 16 * rb;
  int tau = t % 16, chunk = c / 8, w = c % 8;
  *bit = 0;
  if (cfg->qmode == ORC_Q_F16) return base + chunk * 256 + tau * 16 + w * 2;
  int hb = hi_bits(cfg->qmode), lb = lo_bits(cfg->qmode);
  int nhi = orc_outlier_channels(cfg->qmode, r) / 8;
  int bits = chunk < nhi ? hb : lb;
  int64_t cbase = chunk < nhi ? base + chunk * 16 * hb
                              : base + nhi * 16 * hb + (chunk - nhi) * 16 * lb;
  int64_t tok = cbase + tau * bits;            /* the token's 8 codes take `bits` bytes */
  if (bits == 8) return tok + w;
  if (bits == 4) { *bit = 4 * (w % 2); return tok + w / 2; }
  *bit = 3 * w;                                /* 3-bit: the token's 24-bit word */
  return tok;
}

/* Key meta: per 16-token block and group, 16 (s, z) fp16 pairs, one per token.
 * Returns the offset of s; z follows at +2. */
static int64_t key_meta_at(const orc_cfg* cfg, int g, int b, int t, int gi, int64_t* zoff) {
  int ng = orc_n_groups(cfg->qmode, cfg->key_rank[g]);
  int64_t off = orc_plane_offset(cfg, 1, g) +
                ((row_of(cfg, b, t) / 16) * ng + gi) * 64 + (t % 16) * 4;
  *zoff = off + 2;
  return off;
}

/* Value code of channel c at token t.  A 32-token block is split into four
 * 8-token chunks k: the tokens u = 16h + 4j + k (h = 0, 1; j = 0..3) of the
 * block, at slot 4h + j.  Within a precision region the order is
 * [channel][chunk][slots]. */
static void value_slot(int t, int* kq, int* slot) {
  int tau = t % 32, sub = tau / 16, rem = tau % 16;
  *kq = rem % 4;
  *slot = 4 * sub + rem / 4;
}

/* Within a precision region the order is [channel][chunk][slots]; a
 * (channel, chunk) holds its 8 slots in 16 bytes (fp16), 8 bytes (8-bit: slot
 * in byte), 4 bytes (4-bit: slot 2k in nibble k, slot 2k+1 in nibble k+4 of
 * the little-endian 32-bit word) or 3 bytes (3-bit: slot 2k at bits 3k..3k+2,
 * slot 2k+1 at bits 12+3k..14+3k of the little-endian 24-bit word). */
static int64_t value_code_at(const orc_cfg* cfg, int b, int t, int c, int* bit) {
  int r = cfg->value_rank;
  int rb = row_bytes(cfg->qmode, r);
  int64_t base = orc_plane_offset(cfg, 2, 0) + (row_of(cfg, b, t) / 32) * 32 * rb;
  int kq, slot;
  value_slot(t, &kq, &slot);
  *bit = 0;
  if (cfg->qmode == ORC_Q_F16) return base + ((int64_t)c * 4 + kq) * 16 + slot * 2;
  int ro = orc_outlier_channels(cfg->qmode, r);
  int hb = hi_bits(cfg->qmode), lb = lo_bits(cfg->qmode);
  int bits = c < ro ? hb : lb;
  int64_t word = c < ro ? base + ((int64_t)c * 4 + kq) * hb
                        : base + 4 * (int64_t)ro * hb + ((int64_t)(c - ro) * 4 + kq) * lb;
  if (bits == 8) return word + slot;
  int pos = (slot % 2 == 0) ? slot / 2 : slot / 2 + 4;   /* nibble / 3-bit field index */
  if (bits == 4) { *bit = 4 * (pos % 2); return word + pos / 2; }
  *bit = (slot % 2 == 0) ? 3 * (slot / 2) : 12 + 3 * (slot / 2);
  return word;
}

/* Value meta: per 32-token block, group and chunk, the 8 scales of the chunk's
 * slots (16 B) followed by their 8 zeros (16 B).  Returns the offset of s. */
static int64_t value_meta_at(const orc_cfg* cfg, int b, int t, int gi, int64_t* zoff) {
  int ng = orc_n_groups(cfg->qmode, cfg->value_rank);
  int kq, slot;
  value_slot(t, &kq, &slot);
  int64_t off = orc_plane_offset(cfg, 3, 0) +
                (row_of(cfg, b, t) / 32) * ng * 128 + (gi * 4 + kq) * 32 + slot * 2;
  *zoff = off + 16;
  return off;
}

static void put16(uint8_t* p, uint16_t v) { p[0] = (uint8_t)(v & 255); p[1] = (uint8_t)(v >> 8); }
static uint16_t get16(const uint8_t* p) { return (uint16_t)(p[0] | (p[1] << 8)); }

static void put_code(uint8_t* cache, int64_t off, int bit, int bits, uint16_t v) {
  if (bits == 16) { put16(cache + off, v); return; }
  if (bits == 8) { cache[off] = (uint8_t)v; return; }
  int nbytes = bits == 3 ? 3 : 1;              /* the container */
  uint32_t word = 0;
  for (int i = 0; i < nbytes; ++i) word |= (uint32_t)cache[off + i] << (8 * i);
  uint32_t mask = ((1u << bits) - 1) << bit;
  word = (word & ~mask) | (((uint32_t)v << bit) & mask);
  for (int i = 0; i < nbytes; ++i) cache[off + i] = (uint8_t)(word >> (8 * i));
}

static uint16_t get_code(const uint8_t* cache, int64_t off, int bit, int bits) {
  if (bits == 16) return get16(cache + off);
  if (bits == 8) return cache[off];
  int nbytes = bits == 3 ? 3 : 1;
  uint32_t word = 0;
  for (int i = 0; i < nbytes; ++i) word |= (uint32_t)cache[off + i] << (8 * i);
  return (uint16_t)((word >> bit) & ((1u << bits) - 1));
}

static int sum_key_rank(const orc_cfg* cfg) {
  int s = 0;
  for (int g = 0; g < cfg->n_kv_heads; ++g) s += cfg->key_rank[g];
  return s;
}

/* one latent block (key head g, or values when g < 0) of one token */
static void store_block(const orc_cfg* cfg, uint8_t* cache, int g, int b, int t,
                        const uint16_t* x) {
  int r = g >= 0 ? cfg->key_rank[g] : cfg->value_rank;
  uint8_t codes[8192];
  uint16_t s[512], z[512];
  int ng = 0;
  if (cfg->qmode != ORC_Q_F16) ng = orc_quantize_block(cfg->qmode, r, x, codes, s, z);
  for (int c = 0; c < r; ++c) {
    int bits, bit;
    orc_channel_group(cfg->qmode, r, c, &bits);
    int64_t off = g >= 0 ? key_code_at(cfg, g, b, t, c, &bit) : value_code_at(cfg, b, t, c, &bit);
    put_code(cache, off, bit, bits, bits == 16 ? x[c] : codes[c]);
  }
  for (int gi = 0; gi < ng; ++gi) {
    int64_t zoff;
    int64_t soff = g >= 0 ? key_meta_at(cfg, g, b, t, gi, &zoff) : value_meta_at(cfg, b, t, gi, &zoff);
    put16(cache + soff, s[gi]);
    put16(cache + zoff, z[gi]);
  }
}

typedef struct {
  const orc_cfg* cfg;
  uint8_t* cache;
  const uint16_t* latents;
  const int32_t* pos;
  int n_new, b;
} append_job;

static void* append_one_sequence(void* arg) {
  append_job* J = (append_job*)arg;
  const orc_cfg* cfg = J->cfg;
  int width = sum_key_rank(cfg) + cfg->value_rank;
  int b = J->b, n_new = J->n_new;
  const int32_t* pos = J->pos;
  const uint16_t* latents = J->latents;
  uint8_t* cache = J->cache;
  {
    for (int j = 0; j < n_new; ++j) {
      int t = pos[b] + j;
      /* rows outside the cache (or on a page outside the pool) are dropped */
      if (t < 0 || t >= cfg->capacity || row_of(cfg, b, t) < 0) continue;
      const uint16_t* x = latents + ((int64_t)b * n_new + j) * width;
      int off = 0;
      for (int g = 0; g < cfg->n_kv_heads; ++g) {
        store_block(cfg, cache, g, b, t, x + off);
        off += cfg->key_rank[g];
      }
      store_block(cfg, cache, -1, b, t, x + off);
    }
  }
  return NULL;
}

/* Sequences own disjoint cache rows, so they are written by one thread each. */
int orc_append(const orc_cfg* cfg, uint8_t* cache, const uint16_t* latents,
               const int32_t* pos, int n_new) {
  append_job jobs[1024];
  pthread_t th[1024];
  /* one thread per sequence: larger batches are refused, not truncated */
  if (cfg->batch < 0 || cfg->batch > 1024 || n_new < 0) return -1;
  int nb = cfg->batch;
  for (int b = 0; b < nb; ++b) {
    append_job J = {cfg, cache, latents, pos, n_new, b};
    jobs[b] = J;
    pthread_create(&th[b], NULL, append_one_sequence, &jobs[b]);
  }
  for (int b = 0; b < nb; ++b) pthread_join(th[b], NULL);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Down-projection (Sec. 3.2): the latent of a token is x . (Sigma V), one    */
/* column block per KV head for keys and one block for the shared values.   */
/* ------------------------------------------------------------------------ */

int orc_downproj(const orc_cfg* cfg, const uint16_t* x, int x_is_bf16,
                 const uint16_t* A, int n_tok, uint16_t* latents, double* z64) {
  int width = sum_key_rank(cfg) + cfg->value_rank;
  int dm = cfg->d_model;
  for (int n = 0; n < n_tok; ++n) {
    for (int col = 0; col < width; ++col) {
      double acc = 0.0;
      for (int k = 0; k < dm; ++k) {
        uint16_t xv = x[(int64_t)n * dm + k];
        double xd = x_is_bf16 ? orc_bf16_to_double(xv) : orc_f16_to_double(xv);
        acc += xd * orc_bf16_to_double(A[(int64_t)k * width + col]);
      }
      if (z64) z64[(int64_t)n * width + col] = acc;
      latents[(int64_t)n * width + col] = orc_double_to_f16(acc);
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Reading the cache back: dequantized value x-hat = z + code * s (exact in  */
/* fp64).                                                                    */
/* ------------------------------------------------------------------------ */

static void load_block(const orc_cfg* cfg, const uint8_t* cache, int g, int b, int t,
                       double* out) {
  int r = g >= 0 ? cfg->key_rank[g] : cfg->value_rank;
  for (int c = 0; c < r; ++c) {
    int bits, bit;
    int gi = orc_channel_group(cfg->qmode, r, c, &bits);
    int64_t off = g >= 0 ? key_code_at(cfg, g, b, t, c, &bit) : value_code_at(cfg, b, t, c, &bit);
    uint16_t code = get_code(cache, off, bit, bits);
    if (bits == 16) { out[c] = orc_f16_to_double(code); continue; }
    int64_t zoff;
    int64_t soff = g >= 0 ? key_meta_at(cfg, g, b, t, gi, &zoff) : value_meta_at(cfg, b, t, gi, &zoff);
    double s = orc_f16_to_double(get16(cache + soff));
    double z = orc_f16_to_double(get16(cache + zoff));
    out[c] = z + (double)code * s;
  }
}

int orc_read_token(const orc_cfg* cfg, const uint8_t* cache, int b, int t,
                   double* khat, double* vhat) {
  int off = 0;
  for (int g = 0; g < cfg->n_kv_heads; ++g) {
    load_block(cfg, cache, g, b, t, khat + off);
    off += cfg->key_rank[g];
  }
  load_block(cfg, cache, -1, b, t, vhat);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* RoPE, rotate-half form (Sec. 3.3: applied to keys after reconstruction,  */
/* at the key's absolute position).                                         */
/* ------------------------------------------------------------------------ */

void orc_rope(double* v, int d, double t, double theta) {
  int h = d / 2;
  for (int j = 0; j < h; ++j) {
    double inv = pow(theta, -2.0 * j / d);
    double phi = t * inv;
    double c = cos(phi), s = sin(phi);
    double a = v[j], bb = v[j + h];
    v[j] = a * c - bb * s;
    v[j + h] = bb * c + a * s;
  }
}

static int key_row_offset(const orc_cfg* cfg, int g) {
  int off = 0;
  for (int i = 0; i < g; ++i) off += cfg->key_rank[i];
  return off;
}

/* Key reconstruction (Sec. 3.2, head-wise decomposition Sec. 4.3.3):
 * k = K'_g . U_K,g^T, i.e. sum over the head's latent channels of
 * latent value times the row of the up-projection block. */
int orc_reconstruct_key(const orc_cfg* cfg, const uint8_t* cache,
                        const uint16_t* Bk, int b, int g, int t, int rope, double* k) {
  int d = cfg->head_dim, r = cfg->key_rank[g];
  double lat[1024];
  load_block(cfg, cache, g, b, t, lat);
  const uint16_t* B = Bk + (int64_t)key_row_offset(cfg, g) * d;
  for (int j = 0; j < d; ++j) {
    double acc = 0.0;
    for (int i = 0; i < r; ++i) acc += lat[i] * orc_f16_to_double(B[(int64_t)i * d + j]);
    k[j] = acc;
  }
  if (rope) orc_rope(k, d, (double)t, cfg->rope_theta);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Decode attention for the query heads of one (sequence b, KV head g).      */
/*   s_t = q . RoPE_t(k_t) / sqrt(d)               (Sec. 3.1)                */
/*   p_t = exp(s_t - max s), l = sum p_t           (two-pass softmax)        */
/*   a   = sum_t p_t v'_t   over the shared value latent (Sec. 3.3, JD)      */
/*   o   = (a / l) . U_V^T restricted to head g's d output rows (Sec. 3.3)   */
/* Query head i uses KV head floor(i * H_kv / H_q).                          */
/* ------------------------------------------------------------------------ */

typedef struct {
  const orc_cfg* cfg;
  const uint8_t* cache;
  const uint16_t *q, *Bk, *Bv;
  int q_is_bf16;
  const int32_t* ctx_len;
  const unsigned char* want;                   /* [B][H_q] */
  double* out;                                 /* [B][H_q][d], or NULL */
  double* lat;                                 /* [B][H_q][r_v] a/l, or NULL */
  int next_task;                               /* protected by lock */
  pthread_mutex_t lock;
} attn_job;

static void attn_task(attn_job* J, int b, int g) {
  const orc_cfg* cfg = J->cfg;
  int d = cfg->head_dim, Hq = cfg->n_q_heads, Hkv = cfg->n_kv_heads, rv = cfg->value_rank;
  int G = Hq / Hkv;
  int heads[64], nh = 0;
  for (int i = g * G; i < (g + 1) * G; ++i)
    if (J->want[b * Hq + i]) heads[nh++] = i;
  if (nh == 0) return;
  int L = J->ctx_len[b];           /* 0 <= L <= capacity (checked by run_attn) */
  if (L == 0) {
    for (int h = 0; h < nh; ++h) {
      if (J->out)
        for (int j = 0; j < d; ++j) J->out[((int64_t)b * Hq + heads[h]) * d + j] = 0.0;
      if (J->lat)
        for (int c = 0; c < rv; ++c) J->lat[((int64_t)b * Hq + heads[h]) * rv + c] = 0.0;
    }
    return;
  }
  double* qd = malloc(sizeof(double) * nh * d);
  for (int h = 0; h < nh; ++h)
    for (int j = 0; j < d; ++j) {
      uint16_t v = J->q[((int64_t)b * Hq + heads[h]) * d + j];
      qd[h * d + j] = J->q_is_bf16 ? orc_bf16_to_double(v) : orc_f16_to_double(v);
    }
  double* scores = malloc(sizeof(double) * nh * (size_t)L);
  double* k = malloc(sizeof(double) * d);
  double inv_sqrt_d = 1.0 / sqrt((double)d);
  for (int t = 0; t < L; ++t) {
    orc_reconstruct_key(cfg, J->cache, J->Bk, b, g, t, 1, k);
    for (int h = 0; h < nh; ++h) {
      double s = 0.0;
      for (int j = 0; j < d; ++j) s += qd[h * d + j] * k[j];
      scores[(size_t)h * L + t] = s * inv_sqrt_d;
    }
  }
  double* a = calloc((size_t)nh * rv, sizeof(double));
  double* l = calloc(nh, sizeof(double));
  double* v = malloc(sizeof(double) * rv);
  for (int h = 0; h < nh; ++h) {
    double m = -INFINITY;
    for (int t = 0; t < L; ++t) if (scores[(size_t)h * L + t] > m) m = scores[(size_t)h * L + t];
    for (int t = 0; t < L; ++t) scores[(size_t)h * L + t] = exp(scores[(size_t)h * L + t] - m);
  }
  for (int t = 0; t < L; ++t) {
    load_block(cfg, J->cache, -1, b, t, v);
    for (int h = 0; h < nh; ++h) {
      double p = scores[(size_t)h * L + t];
      l[h] += p;
      for (int c = 0; c < rv; ++c) a[(size_t)h * rv + c] += p * v[c];
    }
  }
  int ldv = Hkv * d;
  if (J->lat)
    for (int h = 0; h < nh; ++h)
      for (int c = 0; c < rv; ++c)
        J->lat[((int64_t)b * Hq + heads[h]) * rv + c] = a[(size_t)h * rv + c] / l[h];
  for (int h = 0; h < nh && J->out; ++h) {
    for (int j = 0; j < d; ++j) {
      double o = 0.0;
      for (int c = 0; c < rv; ++c)
        o += (a[(size_t)h * rv + c] / l[h]) * orc_f16_to_double(J->Bv[(int64_t)c * ldv + g * d + j]);
      J->out[((int64_t)b * Hq + heads[h]) * d + j] = o;
    }
  }
  free(qd); free(scores); free(k); free(a); free(l); free(v);
}

static void* attn_worker(void* arg) {
  attn_job* J = (attn_job*)arg;
  int n_tasks = J->cfg->batch * J->cfg->n_kv_heads;
  for (;;) {
    pthread_mutex_lock(&J->lock);
    int task = J->next_task++;
    pthread_mutex_unlock(&J->lock);
    if (task >= n_tasks) break;
    attn_task(J, task / J->cfg->n_kv_heads, task % J->cfg->n_kv_heads);
  }
  return NULL;
}

static int run_attn(const orc_cfg* cfg, const uint8_t* cache, const uint16_t* q,
                    int q_is_bf16, const uint16_t* Bk, const uint16_t* Bv,
                    const int32_t* ctx_len, const int32_t* sel, int n_sel,
                    double* out, double* lat, int n_threads) {
  int Hq = cfg->n_q_heads;
  /* a context longer than the cache (or negative) is an error, not clamped */
  for (int b = 0; b < cfg->batch; ++b)
    if (ctx_len[b] < 0 || ctx_len[b] > cfg->capacity) return -1;
  for (int k = 0; sel && k < n_sel; ++k)
    if (sel[2 * k] < 0 || sel[2 * k] >= cfg->batch || sel[2 * k + 1] < 0 || sel[2 * k + 1] >= Hq)
      return -1;
  unsigned char* want = calloc((size_t)cfg->batch * Hq, 1);
  if (sel) {
    for (int k = 0; k < n_sel; ++k) want[sel[2 * k] * Hq + sel[2 * k + 1]] = 1;
  } else {
    memset(want, 1, (size_t)cfg->batch * Hq);
  }
  attn_job J;
  J.cfg = cfg; J.cache = cache; J.q = q; J.Bk = Bk; J.Bv = Bv; J.q_is_bf16 = q_is_bf16;
  J.ctx_len = ctx_len; J.want = want; J.out = out; J.lat = lat; J.next_task = 0;
  pthread_mutex_init(&J.lock, NULL);
  if (n_threads <= 0) n_threads = (int)sysconf(_SC_NPROCESSORS_ONLN);
  int n_tasks = cfg->batch * cfg->n_kv_heads;
  if (n_threads > n_tasks) n_threads = n_tasks;
  if (n_threads < 1) n_threads = 1;
  pthread_t th[256];
  if (n_threads > 256) n_threads = 256;
  for (int i = 0; i < n_threads; ++i) pthread_create(&th[i], NULL, attn_worker, &J);
  for (int i = 0; i < n_threads; ++i) pthread_join(th[i], NULL);
  pthread_mutex_destroy(&J.lock);
  free(want);
  return n_threads;
}

int orc_decode_attn(const orc_cfg* cfg, const uint8_t* cache, const uint16_t* q,
                    int q_is_bf16, const uint16_t* Bk, const uint16_t* Bv,
                    const int32_t* ctx_len, const int32_t* sel, int n_sel,
                    double* out, int n_threads) {
  return run_attn(cfg, cache, q, q_is_bf16, Bk, Bv, ctx_len, sel, n_sel, out, NULL, n_threads);
}

/* The normalized value latent a_i / l_i of every selected query head: the
 * quantity that the reordering of Sec. 3.3 multiplies by U_V (or, with the
 * weights absorbed, by W_out,i U_V,i) once per query head. */
int orc_decode_latent(const orc_cfg* cfg, const uint8_t* cache, const uint16_t* q,
                      int q_is_bf16, const uint16_t* Bk, const int32_t* ctx_len,
                      const int32_t* sel, int n_sel, double* lat, int n_threads) {
  return run_attn(cfg, cache, q, q_is_bf16, Bk, NULL, ctx_len, sel, n_sel, NULL, lat, n_threads);
}

/* Dense attention (Sec. 3.1) from explicit keys and values; RoPE on keys. */
void orc_dense_attn(int d, int L, const double* q, const double* K,
                    const double* V, double theta, double* out) {
  double* s = malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
  double* k = malloc(sizeof(double) * d);
  double m = -INFINITY;
  for (int t = 0; t < L; ++t) {
    memcpy(k, K + (int64_t)t * d, sizeof(double) * d);
    orc_rope(k, d, (double)t, theta);
    double acc = 0.0;
    for (int j = 0; j < d; ++j) acc += q[j] * k[j];
    s[t] = acc / sqrt((double)d);
    if (s[t] > m) m = s[t];
  }
  double l = 0.0;
  for (int t = 0; t < L; ++t) { s[t] = exp(s[t] - m); l += s[t]; }
  for (int j = 0; j < d; ++j) {
    double acc = 0.0;
    for (int t = 0; t < L; ++t) acc += s[t] * V[(int64_t)t * d + j];
    out[j] = L > 0 ? acc / l : 0.0;
  }
  free(s); free(k);
}
