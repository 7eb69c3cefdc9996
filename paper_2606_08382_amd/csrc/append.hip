// starkv_append kernels (gfx950).
//
// downproj: latents = x . A_all (Sec. 3.2: K' = x (Sigma V)_K per head, V' =
//   x (Sigma V)_V), bf16 operands on v_mfma_f32_16x16x32_bf16, fp32 partial sums
//   per k-split, then a fixed-order reduction rounded to fp16.
// pack: per-token group quantization of every latent block into the cache
//   (Sec. 4.4: an outlier block and an inlier block at b_out > b_in bits: 8/4,
//   4/4, or the paper's 4/3).  The scale is
//   the smallest fp16 not below (max - min)/(2^b - 1) and the codes round half
//   to even; both are evaluated in fp64, which is exact for fp16 operands, so
//   the codes do not depend on evaluation order.
#include <hip/hip_runtime.h>

#include "starkv_internal.h"

namespace starkv {

typedef __bf16 b8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ quantizer math

__device__ __forceinline__ double h2d(uint16_t h) {
  return (double)__builtin_bit_cast(_Float16, h);
}

// Smallest fp16 >= q for finite q > 0, from the exponent and a ceiling of the
// scaled significand (exact: scaling by powers of two is exact in fp64).
__device__ uint16_t f16_ceil_pos(double q) {
  const int e = ilogb(q);
  if (e < -14) {
    const double m = ceil(ldexp(q, 24));            // units of 2^-24; 1024 = smallest normal
    return (uint16_t)m;
  }
  double m = ceil(ldexp(q, 10 - e));                // [1024, 2048]
  int E = e;
  if (m == 2048.0) { m = 1024.0; E += 1; }
  if (E > 15) return 0x7C00;
  return (uint16_t)(((E + 15) << 10) | ((int)m - 1024));
}

struct GroupQ {
  uint16_t s, z;
  double sv, zv, levels;
};

__device__ __forceinline__ GroupQ group_params(const uint16_t* x, int n, int bits) {
  double lo = h2d(x[0]), hi = lo;
  for (int i = 1; i < n; ++i) {
    const double v = h2d(x[i]);
    lo = v < lo ? v : lo;
    hi = v > hi ? v : hi;
  }
  GroupQ g;
  g.levels = (double)((1 << bits) - 1);
  g.z = __builtin_bit_cast(uint16_t, (_Float16)lo);   // lo is an fp16 value
  g.s = (hi > lo) ? f16_ceil_pos((hi - lo) / g.levels) : (uint16_t)0;
  g.sv = h2d(g.s);
  g.zv = lo;
  return g;
}

__device__ __forceinline__ uint32_t group_code(const GroupQ& g, uint16_t x) {
  if (g.sv == 0.0) return 0;
  double c = rint((h2d(x) - g.zv) / g.sv);
  c = c < 0.0 ? 0.0 : (c > g.levels ? g.levels : c);
  return (uint32_t)c;
}

// ------------------------------------------------------------------ pack kernels
// Lanes 32h .. 32h + 31 of a wave hold the channels c0 .. c0 + 31 of one token
// and one quantization group (lanes at or beyond the group's width are off).
// The group's min and max come from reductions within those 32 lanes, the scale
// and the codes from fp64 arithmetic per lane, and a token's key codes are
// packed into its cache words with shuffles.
//
// Two kernels.  Decode-sized appends (one token per wave) first sum the
// down-projection's split-k partials (fixed order) and store the fp16 latent;
// a token then writes its value nibbles into words that hold eight tokens four
// apart, with an atomic AND/OR pair unless each word has one writer.  Appends
// given as fp16 latents take one wave per 32-row block of a sequence and
// group, with lane (h, c) on channel c0 + c of the block's tokens 2i + h: every
// value word of the block is then assembled in one lane and stored once.

__device__ __forceinline__ float wave_min32(float v) {
  for (int o = 16; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_max32(float v) {
  for (int o = 16; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

struct PackGroup {
  int bl, gi, c0, n, bits, ro, hb, lb, ngr, rb;
  bool is_v;
};

// The quantization group of work item `item`: its block (a key head or the
// value latent), region, channels c0 .. c0 + n - 1 of the block and bit width.
__device__ __forceinline__ PackGroup make_group(const AppendParams& p, int item) {
  PackGroup G;
  G.bl = p.item_block[item];
  G.gi = p.item_group[item];
  const int r = p.rank[G.bl];
  G.ro = p.ro[G.bl];
  G.is_v = (G.bl == p.n_kv);
  G.ngr = p.ng[G.bl];
  G.rb = p.row_bytes[G.bl];
  // bits of the outlier (hb) and inlier (lb) regions
  G.hb = p.qmode == STARKV_Q_MIX8_4 ? 8 : 4;
  G.lb = p.qmode == STARKV_Q_MIX4_3 ? 3 : 4;
  if (p.qmode == STARKV_Q_F16) {
    G.c0 = 32 * G.gi; G.n = min(32, r - G.c0); G.bits = 16;
  } else {
    const int ngo = (G.ro + 31) / 32;
    if (G.gi < ngo) { G.c0 = 32 * G.gi; G.n = min(32, G.ro - G.c0); G.bits = G.hb; }
    else { G.c0 = G.ro + 32 * (G.gi - ngo); G.n = min(32, r - G.c0); G.bits = G.lb; }
  }
  return G;
}

// Scale, zero and the lane's code for one token of a group (bits < 16); `on`
// says whether the lane holds one of the group's channels.  The reductions run
// over the 32 lanes of the lane's half.
struct QCode {
  uint16_t s16, z16;
  uint32_t code;
};

__device__ __forceinline__ QCode quantize_lane(uint16_t xb, bool on, int bits) {
  // the fp16 values compare exactly in fp32
  const float xf = (float)__builtin_bit_cast(_Float16, xb);
  const float lo = wave_min32(on ? xf : INFINITY);
  const float hi = wave_max32(on ? xf : -INFINITY);
  const double levels = (double)((1 << bits) - 1);
  QCode q;
  q.s16 = (hi > lo) ? f16_ceil_pos(((double)hi - (double)lo) / levels) : (uint16_t)0;
  q.z16 = __builtin_bit_cast(uint16_t, (_Float16)lo);
  const double sv = h2d(q.s16);
  q.code = 0;
  if (sv != 0.0) {
    double c = rint(((double)xf - (double)lo) / sv);
    c = c < 0.0 ? 0.0 : (c > levels ? levels : c);
    q.code = (uint32_t)c;
  }
  if (!on) q.code = 0;
  return q;
}

// A token's key codes and meta (rows in 16-token blocks: kblk, tau).  cl is
// the lane's index in its 32-lane half; the writers are `on` lanes leading
// groups of 4 (8-bit) or 8 (4-, 3-bit) channels, and the meta is written when
// `meta` is set (by one lane).
__device__ __forceinline__ void store_key_token(const AppendParams& p, const PackGroup& G, int cl,
                                                int64_t kblk, int tau, const QCode& q, bool on,
                                                bool meta) {
  const int c = G.c0 + cl, bits = G.bits, hb = G.hb, lb = G.lb;
  uint8_t* kb = p.cache + p.code_off[G.bl] + kblk * 16 * G.rb;
  const int nhi = G.ro / 8;              // outlier chunks (16 tokens x hb bytes each)
  const int ch = c / 8;
  uint8_t* chunk = ch < nhi ? kb + ch * 16 * hb : kb + nhi * 16 * hb + (ch - nhi) * 16 * lb;
  if (bits == 8) {          // 4 codes per 32-bit word, lanes 4k..4k+3
    uint32_t wv = q.code << (8 * (cl & 3));
    wv |= __shfl_xor(wv, 1);
    wv |= __shfl_xor(wv, 2);
    if (on && (cl & 3) == 0)
      *reinterpret_cast<uint32_t*>(chunk + tau * 8 + (c % 8)) = wv;
  } else {                  // a token's 8 codes of a chunk, lanes 8k..8k+7: channel
    // w at bits bits*w (4-bit: one 32-bit word; 3-bit: 3 bytes, stored bytewise
    // since neighbouring tokens share 32-bit words)
    uint32_t wv = q.code << (bits * (cl & 7));
    wv |= __shfl_xor(wv, 1);
    wv |= __shfl_xor(wv, 2);
    wv |= __shfl_xor(wv, 4);
    if (on && (cl & 7) == 0) {
      if (bits == 4) {
        *reinterpret_cast<uint32_t*>(chunk + tau * 4) = wv;
      } else {
        uint8_t* d = chunk + tau * 3;
        d[0] = (uint8_t)wv;
        d[1] = (uint8_t)(wv >> 8);
        d[2] = (uint8_t)(wv >> 16);
      }
    }
  }
  if (meta) {
    uint16_t* m = reinterpret_cast<uint16_t*>(p.cache + p.meta_off[G.bl] +
                                              (kblk * G.ngr + G.gi) * 64 + tau * 4);
    m[0] = q.s16;
    m[1] = q.z16;
  }
}

// Value words of a 32-row block: the outlier region's (channel, chunk) words of
// 8 bytes first, then the inlier region's of lb bytes; chunk kq holds the
// block's tokens u = kq + 4 j in slots 4 (u / 16) + (u % 16) / 4.
__device__ __forceinline__ int64_t value_word(const PackGroup& G, int c, int kq) {
  return c < G.ro ? ((int64_t)c * 4 + kq) * G.hb
                  : 4LL * G.ro * G.hb + ((int64_t)(c - G.ro) * 4 + kq) * G.lb;
}
// bit offset of slot `slot` in a 4-bit (32-bit word) or 3-bit (24-bit word)
// value word: slot 2k at field k, slot 2k + 1 at field k + 4
__device__ __forceinline__ int value_shift(int bits, int slot) {
  return bits == 4 ? ((slot % 2 == 0) ? 4 * (slot / 2) : 16 + 4 * (slot / 2))
                   : ((slot % 2 == 0) ? 3 * (slot / 2) : 12 + 3 * (slot / 2));
}

// One token of a decode-sized append (lane i: channel c0 + i, lanes 32..63 off).
__device__ __forceinline__ void pack_token(const AppendParams& p, const PackGroup& G, int lane,
                                           int b, int t, uint16_t xb) {
  const int bits = G.bits;
  const bool on = lane < G.n;
  const int c = G.c0 + lane;
  if (t < 0 || t >= p.capacity) return;     // rows outside the cache are dropped
  if (p.rmap.table) {                        // and rows on pages outside the pool
    const int pg = p.rmap.table[(int64_t)b * p.rmap.per_seq + (t >> p.rmap.shift)];
    if (pg < 0 || pg >= p.rmap.n_pages) return;
  }
  uint8_t* code_plane = p.cache + p.code_off[G.bl];
  uint8_t* meta_plane = p.cache + p.meta_off[G.bl];
  const int64_t row = cache_row(p.rmap, b, t);
  const int64_t kblk = row / 16;
  const int tau = t % 16;
  const int64_t vblk = row / 32;
  const int u = t % 32, kq = u % 4, slot = 4 * (u / 16) + (u % 16) / 4;
  if (bits == 16) {
    if (on) {
      if (!G.is_v)
        *reinterpret_cast<uint16_t*>(code_plane + kblk * 16 * G.rb + (c / 8) * 256 + tau * 16 + (c % 8) * 2) = xb;
      else
        *reinterpret_cast<uint16_t*>(code_plane + vblk * 32 * G.rb + ((int64_t)c * 4 + kq) * 16 + slot * 2) = xb;
    }
    return;
  }
  const QCode q = quantize_lane(xb, on, bits);
  if (!G.is_v) {
    store_key_token(p, G, lane, kblk, tau, q, on, lane == 0);
    return;
  }
  uint8_t* vb = code_plane + vblk * 32 * G.rb;
  if (on) {
    const int64_t word = value_word(G, c, kq);
    if (bits == 8) {
      vb[word + slot] = (uint8_t)q.code;
    } else {
      // tokens of one launch own disjoint fields, updated with atomic AND/OR on
      // the aligned 32-bit word(s) holding them (a 3-bit field may straddle two)
      const uint64_t abit = (uint64_t)((vb + word) - p.cache) * 8 + value_shift(bits, slot);
      unsigned int* wp = reinterpret_cast<unsigned int*>(p.cache) + abit / 32;
      const int s0 = (int)(abit % 32);
      const uint32_t fmask = (1u << bits) - 1;
      if (p.single_writer && bits == 4) {
        // at most four new tokens per sequence: every 4-bit word (eight tokens
        // four apart) has one writer in this launch
        *wp = (*wp & ~(fmask << s0)) | (q.code << s0);
      } else {
        atomicAnd(wp, ~(fmask << s0));
        atomicOr(wp, q.code << s0);
        if (s0 + bits > 32) {                // the field's high bits in the next word
          atomicAnd(wp + 1, ~(fmask >> (32 - s0)));
          atomicOr(wp + 1, q.code >> (32 - s0));
        }
      }
    }
  }
  if (lane == 0) {
    uint16_t* m = reinterpret_cast<uint16_t*>(meta_plane + (vblk * G.ngr + G.gi) * 128 + kq * 32 + slot * 2);
    m[0] = q.s16;
    m[8] = q.z16;
  }
}

// Decode-sized appends: one token per wave, its latents summed from the
// down-projection's split-k partials in a fixed order (up to 64 loads in
// flight) and stored as fp16 before the pack.
__global__ __launch_bounds__(256) void pack_kernel(AppendParams p) {
  const int lane = threadIdx.x & 63;
  const int wid = blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
  const int n_tok = p.batch * p.n_new;
  if (wid >= n_tok * p.n_items) return;
  const int tok = wid / p.n_items, item = wid % p.n_items;
  const PackGroup G = make_group(p, item);
  const bool on = lane < G.n;
  const int c = G.c0 + lane;
  const int pos = p.pos[tok / p.n_new];
  uint16_t xb = 0;
  if (on) {
    const int64_t li = (int64_t)tok * p.width + p.lat_off[G.bl] + c;
    const int64_t mn = (int64_t)n_tok * p.width;
    float acc = 0.0f;
    int k = 0;
    for (; k + 64 <= p.k_split; k += 64) {
      float v[64];
#pragma unroll
      for (int u = 0; u < 64; ++u) v[u] = p.partial[(k + u) * mn + li];
#pragma unroll
      for (int u = 0; u < 64; ++u) acc += v[u];
    }
    for (; k + 16 <= p.k_split; k += 16) {
      float v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = p.partial[(k + u) * mn + li];
#pragma unroll
      for (int u = 0; u < 16; ++u) acc += v[u];
    }
    for (; k < p.k_split; ++k) acc += p.partial[k * mn + li];
    xb = __builtin_bit_cast(uint16_t, (_Float16)acc);
    p.lat_out[li] = xb;
  }
  const int b = tok / p.n_new, j = tok % p.n_new;
  pack_token(p, G, lane, b, pos + j, xb);
}

// Appends given as fp16 latents: one wave per (sequence, 32-row block that the
// rows pos .. pos + n_new - 1 touch, group).  A 3- or 4-bit value word of the
// block (eight tokens of one channel, four apart) belongs to one lane, which
// assembles the new fields and stores the word once, reading it first only
// when the append covers part of it; no other wave of the launch writes it.
__global__ __launch_bounds__(256) void pack_block_kernel(AppendParams p) {
  const int lane = threadIdx.x & 63;
  const int wid = blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
  const int nblk = (p.n_new + 31) / 32 + 1;     // blocks a run of n_new rows can touch
  const int per_seq = nblk * p.n_items;
  if (wid >= p.batch * per_seq) return;
  const int b = wid / per_seq, rem = wid % per_seq;
  const int bi = rem / p.n_items, item = rem % p.n_items;
  const int t0 = p.pos[b];
  const int a = (t0 >> 5) + bi;                 // rows 32 a .. 32 a + 31 of the sequence
  // rows outside the cache are dropped
  const int t_lo = max(max(t0, 32 * a), 0);
  const int t_hi = min(min(t0 + p.n_new, 32 * a + 32), p.capacity);
  if (t_lo >= t_hi) return;
  if (p.rmap.table) {                           // and rows on pages outside the pool
    const int pg = p.rmap.table[(int64_t)b * p.rmap.per_seq + ((32 * a) >> p.rmap.shift)];
    if (pg < 0 || pg >= p.rmap.n_pages) return;
  }
  const PackGroup G = make_group(p, item);
  const int h = lane >> 5, cl = lane & 31;
  const bool on = cl < G.n;
  const int c = G.c0 + cl;
  const int bits = G.bits;
  const int64_t row0 = cache_row(p.rmap, b, 32 * a);   // 32-aligned: pages hold >= 128 rows
  // the lane's 16 latents (tokens u = 2 i + h of the block), loaded together
  uint16_t xb[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int t = 32 * a + 2 * i + h;
    xb[i] = 0;
    if (on && t >= t_lo && t < t_hi)
      xb[i] = p.lat[((int64_t)b * p.n_new + (t - t0)) * p.width + p.lat_off[G.bl] + c];
  }
  uint8_t* code_plane = p.cache + p.code_off[G.bl];
  uint8_t* meta_plane = p.cache + p.meta_off[G.bl];
  uint8_t* vb = code_plane + (row0 / 32) * 32 * G.rb;
  // value words of chunks kq = h and kq = h + 2 (3- and 4-bit): new fields, and
  // the bits they cover
  uint32_t acc[2] = {0u, 0u}, cov[2] = {0u, 0u};
  const uint32_t fmask = bits < 16 ? (1u << bits) - 1 : 0u;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int u = 2 * i + h, t = 32 * a + u;
    const bool live = t >= t_lo && t < t_hi;    // uniform in the lane's half
    const int64_t kblk = (row0 + u) / 16;
    const int tau = u % 16, kq = u % 4, slot = 4 * (u / 16) + (u % 16) / 4;
    if (bits == 16) {
      if (on && live) {
        if (!G.is_v)
          *reinterpret_cast<uint16_t*>(code_plane + kblk * 16 * G.rb + (c / 8) * 256 + tau * 16 + (c % 8) * 2) = xb[i];
        else
          *reinterpret_cast<uint16_t*>(vb + ((int64_t)c * 4 + kq) * 16 + slot * 2) = xb[i];
      }
      continue;
    }
    const QCode q = quantize_lane(xb[i], on, bits);
    if (!G.is_v) {
      store_key_token(p, G, cl, kblk, tau, q, on && live, live && cl == 0);
      continue;
    }
    if (on && live) {
      if (bits == 8) {
        vb[value_word(G, c, kq) + slot] = (uint8_t)q.code;
      } else {
        const int sh = value_shift(bits, slot);
        acc[i & 1] |= q.code << sh;
        cov[i & 1] |= fmask << sh;
      }
    }
    if (live && cl == 0) {
      uint16_t* m = reinterpret_cast<uint16_t*>(meta_plane + ((row0 / 32) * G.ngr + G.gi) * 128 +
                                                kq * 32 + slot * 2);
      m[0] = q.s16;
      m[8] = q.z16;
    }
  }
  if (G.is_v && on && (bits == 4 || bits == 3)) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {               // chunk kq = 2 k + h
      if (cov[k] == 0u) continue;
      uint8_t* wd = vb + value_word(G, c, 2 * k + h);
      if (bits == 4) {
        uint32_t* w32 = reinterpret_cast<uint32_t*>(wd);
        *w32 = cov[k] == 0xFFFFFFFFu ? acc[k] : ((*w32 & ~cov[k]) | acc[k]);
      } else {                                  // 24-bit word, bytewise (not aligned)
        uint32_t old = 0u;
        if (cov[k] != 0xFFFFFFu) old = (uint32_t)wd[0] | ((uint32_t)wd[1] << 8) | ((uint32_t)wd[2] << 16);
        const uint32_t v = (old & ~cov[k]) | acc[k];
        wd[0] = (uint8_t)v;
        wd[1] = (uint8_t)(v >> 8);
        wd[2] = (uint8_t)(v >> 16);
      }
    }
  }
}

// ------------------------------------------------------------------ down-projection
// Split-k tiles of 64 rows x 64 columns; each workgroup covers k_chunk (a
// multiple of BK) of K in steps of BK = kDownprojK = 128, so a decode-sized
// append costs one or two rounds of loads per workgroup.  Per step, thread t
// loads four 16-byte vectors of A_all (k rows t/8 + 32 i, columns 8 (t%8)..)
// and four of x (rows t/16 + 16 i, k 8 (t%16)..); A is stored transposed.
constexpr int BM = 64, BN = 64, BK = kDownprojK;

__global__ __launch_bounds__(256) void downproj_kernel(DownprojParams p) {
  __shared__ __align__(16) __bf16 xs[BM][BK + 8];
  __shared__ __align__(16) __bf16 as[BN][BK + 8];    // transposed A tile: [n][k]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM, ks = blockIdx.z;
  const int k_lo = ks * p.k_chunk;
  const int k_hi = min(p.k, k_lo + p.k_chunk);
  const int wm = (w >> 1) * 32, wn = (w & 1) * 32;
  const bool vec_a = (p.n & 7) == 0;                 // 16-byte rows of A_all
  f4 acc[2][2];
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j) acc[i][j] = (f4){0, 0, 0, 0};
  for (int k0 = k_lo; k0 < k_hi; k0 += BK) {
    u4 xv[4], av[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {         // x: rows tid/16 + 16 i, k 8 (tid%16) ..
      const int r = tid / 16 + 16 * i, kk = (tid % 16) * 8;
      const int m = m0 + r, k = k0 + kk;
      xv[i] = (u4){0, 0, 0, 0};
      if (m < p.m && k + 8 <= k_hi) {
        xv[i] = *reinterpret_cast<const u4*>(p.x + (int64_t)m * p.k + k);
      } else if (m < p.m) {
        uint16_t tmp[8];
        for (int e = 0; e < 8; ++e) tmp[e] = (k + e < k_hi) ? p.x[(int64_t)m * p.k + k + e] : (uint16_t)0;
        xv[i] = *reinterpret_cast<u4*>(tmp);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {         // A: k rows tid/8 + 32 i, columns 8 (tid%8) ..
      const int kr = tid / 8 + 32 * i, nn = (tid % 8) * 8;
      const int k = k0 + kr, n = n0 + nn;
      av[i] = (u4){0, 0, 0, 0};
      if (k < k_hi && vec_a && n + 8 <= p.n) {
        av[i] = *reinterpret_cast<const u4*>(p.a + (int64_t)k * p.n + n);
      } else if (k < k_hi) {
        uint16_t tmp[8];
        for (int e = 0; e < 8; ++e) tmp[e] = (n + e < p.n) ? p.a[(int64_t)k * p.n + n + e] : (uint16_t)0;
        av[i] = *reinterpret_cast<u4*>(tmp);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<u4*>(&xs[tid / 16 + 16 * i][(tid % 16) * 8]) = xv[i];
      const int kr = tid / 8 + 32 * i, nn = (tid % 8) * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        as[nn + e][kr] = __builtin_bit_cast(__bf16, (uint16_t)(av[i][e / 2] >> (16 * (e & 1))));
    }
    __syncthreads();
    const int row = lane & 15, kq = lane >> 4;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      b8 af[2], bf[2];
      for (int i = 0; i < 2; ++i) af[i] = *reinterpret_cast<const b8*>(&xs[wm + 16 * i + row][kk + 8 * kq]);
      for (int j = 0; j < 2; ++j) bf[j] = *reinterpret_cast<const b8*>(&as[wn + 16 * j + row][kk + 8 * kq]);
      for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  // C tile (16x16): lane holds rows 4*(lane/16)+e of column lane%16
  const int cn = lane & 15, rq = lane >> 4;
  float* out = p.partial + (int64_t)ks * p.m * p.n;
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j)
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + wm + 16 * i + 4 * rq + e;
        const int n = n0 + wn + 16 * j + cn;
        if (m < p.m && n < p.n) out[(int64_t)m * p.n + n] = acc[i][j][e];
      }
}

// Down-projection for a few rows (decode appends): A_all is streamed once with
// 16-byte loads.  Workgroup = (128 columns, 64 rows of k): thread (kg, cg)
// takes rows 4*kg..4*kg+3 and columns 8*cg..8*cg+7; the sixteen k groups meet
// in LDS and one fp32 partial per k block is written.
constexpr int kSmallCols = 128, kSmallK = 64;

__global__ __launch_bounds__(256) void downproj_small_kernel(DownprojParams p) {
  extern __shared__ __align__(16) float dsm[];     // [16][M][kSmallCols]
  __shared__ __align__(16) uint16_t xs[kSmallM][kSmallK];
  const int tid = threadIdx.x, cg = tid % 16, kg = tid / 16;
  const int n0 = blockIdx.x * kSmallCols + 8 * cg;
  const int k0 = blockIdx.y * kSmallK;
  const int M = p.m;
  // A rows first (clamped addresses, zeroed afterwards), then the few x values
  u4 av[4];
  {
    const int nc = min(n0, p.n - 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = min(k0 + 4 * kg + i, p.k - 1);
      av[i] = *reinterpret_cast<const u4*>(p.a + (int64_t)k * p.n + nc);
    }
  }
  for (int i = tid; i < M * kSmallK; i += 256) {
    const int m = i / kSmallK, kk = i % kSmallK;
    xs[m][kk] = (k0 + kk < p.k) ? p.x[(int64_t)m * p.k + k0 + kk] : (uint16_t)0;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (k0 + 4 * kg + i >= p.k || n0 >= p.n) av[i] = (u4){0, 0, 0, 0};
  __syncthreads();
  float acc[kSmallM][8];
#pragma unroll
  for (int m = 0; m < kSmallM; ++m)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[m][e] = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float a[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      a[2 * e] = __uint_as_float(av[i][e] << 16);
      a[2 * e + 1] = __uint_as_float(av[i][e] & 0xFFFF0000u);
    }
#pragma unroll
    for (int m = 0; m < kSmallM; ++m) {
      if (m < M) {
        const float xv = __uint_as_float((uint32_t)xs[m][4 * kg + i] << 16);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[m][e] = __builtin_fmaf(xv, a[e], acc[m][e]);
      }
    }
  }
#pragma unroll
  for (int m = 0; m < kSmallM; ++m)
    if (m < M) {
      f4* d = reinterpret_cast<f4*>(dsm + ((kg * M + m) * kSmallCols + 8 * cg));
      d[0] = (f4){acc[m][0], acc[m][1], acc[m][2], acc[m][3]};
      d[1] = (f4){acc[m][4], acc[m][5], acc[m][6], acc[m][7]};
    }
  __syncthreads();
  float* out = p.partial + (int64_t)blockIdx.y * p.m * p.n;
  for (int i = tid; i < M * kSmallCols; i += 256) {
    const int m = i / kSmallCols, c = i % kSmallCols;
    const int n = blockIdx.x * kSmallCols + c;
    if (n < p.n) {
      float v = 0.0f;
#pragma unroll
      for (int g = 0; g < 16; ++g) v += dsm[(g * M + m) * kSmallCols + c];
      out[(int64_t)m * p.n + n] = v;
    }
  }
}

// ------------------------------------------------------------------ prefill down-projection
// Large appends (a prefill): Z = X . A_all as one GEMM.  A_all [K][N] is first
// transposed into the workspace (At [N][K]), so that both operands are
// k-contiguous; the GEMM accumulates all of K in fp32 on
// v_mfma_f32_16x16x32_bf16 and writes the fp16 latents directly (one rounding,
// as the split-k path's pack does).  A workgroup of WMW x WNW waves computes a
// (64 WMW) x (TN WNW) tile, each wave 64 x TN; k steps of 64 are staged in LDS
// with a padded row (conflict-free 16-byte reads), double buffered: the next
// step's global loads are in flight while the current step's MFMAs run.  Large
// problems take 256 x 192 tiles of eight 64 x 96 waves (LDS traffic per flop a
// third lower than with 64 x 48 waves), smaller ones 128 x 96 tiles of four
// waves.
constexpr int GK = 64, GKP = GK + 8;

__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* a, uint16_t* at,
                                                             int K, int N) {
  __shared__ uint16_t t[64][66];
  const int k0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  for (int i = threadIdx.x; i < 64 * 64; i += 256) {
    const int r = i / 64, c = i % 64;             // r: k, c: n (coalesced reads)
    const int k = k0 + r, n = n0 + c;
    t[r][c] = (k < K && n < N) ? a[(int64_t)k * N + n] : (uint16_t)0;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 64 * 64; i += 256) {
    const int r = i / 64, c = i % 64;             // r: n, c: k (coalesced writes)
    const int n = n0 + r, k = k0 + c;
    if (n < N && k < K) at[(int64_t)n * K + k] = t[c][r];
  }
}

template <int WMW, int WNW, int TN>
__global__ __launch_bounds__(64 * WMW * WNW) void gemm_bf16_nt_kernel(DownprojParams p) {
  constexpr int NTH = 64 * WMW * WNW;             // threads
  constexpr int GM = 64 * WMW, GN = TN * WNW;     // workgroup tile
  constexpr int NT = TN / 16;                     // 16-column tiles per wave
  constexpr int NA = GM * GK / 8 / NTH;           // 16-byte chunks of the X tile per thread
  constexpr int NB = GN * GK / 8 / NTH;           // 16-byte chunks of the B tile per thread
  static_assert(NA * NTH == GM * GK / 8 && NB * NTH == GN * GK / 8, "whole chunks per thread");
  __shared__ __align__(16) uint16_t xs[2][GM * GKP];
  __shared__ __align__(16) uint16_t bs[2][GN * GKP];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int M = p.m, N = p.n, K = p.k;            // K is a multiple of GK (checked by the host)
  // workgroups are dealt to the eight XCDs in turn (workgroup i on XCD i % 8):
  // tiles are numbered row-major and XCD x takes a contiguous run of them, so
  // the column tiles of a row of X share that XCD's L2
  const int n_ct = (N + GN - 1) / GN, n_t = n_ct * ((M + GM - 1) / GM);
  const int per_xcd = (n_t + 7) / 8;
  const int t = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t >= n_t) return;
  const int n0 = (t % n_ct) * GN, m0 = (t / n_ct) * GM;
  const int wm = (w / WNW) * 64, wn = (w % WNW) * TN;
  // global -> register staging: chunk c = tid + NTH i of a (rows x 64) tile is
  // row c / 8, k chunk c % 8 (16 bytes); rows past M or N read the last row
  u4 rx[NA], rb[NB];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int c = tid + NTH * i, row = c >> 3, kc = c & 7;
      const int m = min(m0 + row, M - 1);
      rx[i] = *reinterpret_cast<const u4*>(p.x + (int64_t)m * K + k0 + 8 * kc);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int c = tid + NTH * i, row = c >> 3, kc = c & 7;
      const int n = min(n0 + row, N - 1);
      rb[i] = *reinterpret_cast<const u4*>(p.at + (int64_t)n * K + k0 + 8 * kc);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int c = tid + NTH * i, row = c >> 3, kc = c & 7;
      *reinterpret_cast<u4*>(&xs[buf][row * GKP + 8 * kc]) = rx[i];
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int c = tid + NTH * i, row = c >> 3, kc = c & 7;
      *reinterpret_cast<u4*>(&bs[buf][row * GKP + 8 * kc]) = rb[i];
    }
  };
  f4 acc[4][NT];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = (f4){0, 0, 0, 0};
  const int nk = K / GK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int fr = lane & 15, fk = 8 * (lane >> 4);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * GK);
#pragma unroll
    for (int kk = 0; kk < GK; kk += 32) {
      b8 af[4], bf[NT];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const b8*>(&xs[buf][(wm + 16 * i + fr) * GKP + kk + fk]);
#pragma unroll
      for (int j = 0; j < NT; ++j)
        bf[j] = *reinterpret_cast<const b8*>(&bs[buf][(wn + 16 * j + fr) * GKP + kk + fk]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }
  // C tile (16 x 16): lane holds rows 4*(lane/16)+e of column lane%16
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + wm + 16 * i + 4 * (lane >> 4) + e;
        const int n = n0 + wn + 16 * j + fr;
        if (m < M && n < N)
          p.lat[(int64_t)m * N + n] = __builtin_bit_cast(uint16_t, (_Float16)acc[i][j][e]);
      }
}

// The large-problem tile (256 x 192) with its operands copied from global
// memory straight into LDS (global_load_lds, 16 bytes per lane) instead of
// through registers, which leaves registers for sixteen waves of 64 x 48 (four
// per SIMD: the other waves hide each one's fragment reads and the step's
// barrier, worth a third of the GEMM time against two per SIMD): unpadded
// 128-byte rows of 64 k whose
// 16-byte chunk c sits in slot c ^ (row % 8), each lane of a copy fetching the
// chunk that lands where the swizzle wants it, so that a fragment read (one
// chunk of 16 rows) covers eight distinct slots per eight lanes.  Two stages;
// the next step's copies are issued at the start of a step.
constexpr int GDM = 256, GDN = 192, GDWN = 4;   // 16 waves of 64 x 48: four per SIMD
constexpr int GDA = GDM / 8, GDB = GDN / 8;       // 1 KiB copies per k step (A, B)
constexpr int GDSTAGE = (GDM + GDN) * 128;

// WN waves across the 192 columns (tiles of 192 / WN), four across the rows.
template <int WN>
__global__ __launch_bounds__(256 * WN) void gemm_bf16_nt_dma_kernel(DownprojParams p) {
  constexpr int NW = 4 * WN, TN = GDN / WN, NT = TN / 16;
  __shared__ __align__(16) uint8_t sm[2 * GDSTAGE];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int M = p.m, N = p.n, K = p.k;            // K is a multiple of GK (checked by the host)
  // tiles row-major, a contiguous run per XCD (workgroup i on XCD i % 8)
  const int n_ct = (N + GDN - 1) / GDN, n_t = n_ct * ((M + GDM - 1) / GDM);
  const int per_xcd = (n_t + 7) / 8;
  const int t = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t >= n_t) return;
  const int n0 = (t % n_ct) * GDN, m0 = (t / n_ct) * GDM;
  const int wm = (w / WN) * 64, wn = (w % WN) * TN;
  // copy j of a k step: rows 8 j' .. 8 j' + 7 of the A tile (j < GDA) or of the
  // B tile (j' = j - GDA); lane l fills slot l % 8 of row l / 8 with the global
  // chunk (l % 8) ^ (l / 8)
  const int crow = lane >> 3, cchunk = (lane & 7) ^ crow;
  auto issue = [&](int k0, int buf) {
    uint8_t* st = sm + buf * GDSTAGE;
    for (int j = w; j < GDA + GDB; j += NW) {
      const uint16_t* src;
      if (j < GDA) src = p.x + (int64_t)min(m0 + 8 * j + crow, M - 1) * K;
      else src = p.at + (int64_t)min(n0 + 8 * (j - GDA) + crow, N - 1) * K;
      __builtin_amdgcn_global_load_lds(src + k0 + 8 * cchunk, st + j * 1024, 16, 0, 0);
    }
  };
  const int fr = lane & 15, kq = lane >> 4;
  f4 acc[4][NT];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = (f4){0, 0, 0, 0};
  const int nk = K / GK;
  issue(0, 0);
  __builtin_amdgcn_s_waitcnt(0x0F70);               // vmcnt(0)
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) issue((kt + 1) * GK, buf ^ 1);
    const uint8_t* sa = sm + buf * GDSTAGE;
    const uint8_t* sb = sa + GDM * 128;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {                 // 32 k each: chunks 4 kk + kq
      const int c = 4 * kk + kq;
      b8 af[4], bf[NT];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wm + 16 * i + fr;
        af[i] = *reinterpret_cast<const b8*>(sa + r * 128 + ((c ^ (r & 7)) << 4));
      }
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int r = wn + 16 * j + fr;
        bf[j] = *reinterpret_cast<const b8*>(sb + r * 128 + ((c ^ (r & 7)) << 4));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);             // this wave's copies of the next step
    __syncthreads();                                 // every wave's; buf is free
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + wm + 16 * i + 4 * kq + e;
        const int n = n0 + wn + 16 * j + fr;
        if (m < M && n < N)
          p.lat[(int64_t)m * N + n] = __builtin_bit_cast(uint16_t, (_Float16)acc[i][j][e]);
      }
}

// ------------------------------------------------------------------ launchers
int launch_append_pack(const AppendParams& p, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  int64_t waves;
  if (p.partial) {
    waves = (int64_t)p.batch * p.n_new * p.n_items;
    hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, st, p);
  } else {
    waves = (int64_t)p.batch * ((p.n_new + 31) / 32 + 1) * p.n_items;
    hipLaunchKernelGGL(pack_block_kernel, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, st, p);
  }
  return (int)hipGetLastError();
}

int launch_downproj(const DownprojParams& p, void* stream) {
  if (p.at) {                       // the prefill GEMM: transpose A_all, then one pass over K
    if (p.k % GK) return (int)hipErrorInvalidValue;
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(transpose_bf16_kernel, dim3((p.n + 63) / 64, (p.k + 63) / 64), dim3(256), 0,
                       st, p.a, p.at, p.k, p.n);
    // 256 x 192 tiles when they give at least 96 workgroups (one per CU),
    // else 128 x 96 tiles (then at most 4 x 96 of them: a single round at two
    // workgroups per CU)
    if (((p.m + 255) / 256) * ((p.n + 191) / 192) >= 96)
      hipLaunchKernelGGL((gemm_bf16_nt_dma_kernel<GDWN>),
                         dim3(8 * ((((p.n + 191) / 192) * ((p.m + 255) / 256) + 7) / 8)), dim3(256 * GDWN), 0, st, p);
    else
      hipLaunchKernelGGL((gemm_bf16_nt_kernel<2, 2, 48>),
                         dim3(8 * ((((p.n + 95) / 96) * ((p.m + 127) / 128) + 7) / 8)),
                         dim3(256), 0, st, p);
    return (int)hipGetLastError();
  }
  if (p.m <= kSmallM) {
    dim3 grid((p.n + kSmallCols - 1) / kSmallCols, p.k_split);
    const size_t lds = (size_t)16 * p.m * kSmallCols * sizeof(float);
    hipLaunchKernelGGL(downproj_small_kernel, grid, dim3(256), lds,
                       static_cast<hipStream_t>(stream), p);
    return (int)hipGetLastError();
  }
  dim3 grid((p.n + BN - 1) / BN, (p.m + BM - 1) / BM, p.k_split);
  hipLaunchKernelGGL(downproj_kernel, grid, dim3(256), 0, static_cast<hipStream_t>(stream), p);
  return (int)hipGetLastError();
}

}  // namespace starkv
