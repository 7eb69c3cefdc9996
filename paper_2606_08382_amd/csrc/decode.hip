// Decode attention read from the low-rank, quantized cache (gfx950).
//
// decode_split: one workgroup per (context split, sequence, KV-head group), eight
//   waves: four token groups (32 tokens of every 128-token step each, two
//   16-token subtiles) times two halves of the group's KV heads.  For every KV
//   head of its half a wave
//     - dequantizes the key latents of its tokens into MFMA operands (registers),
//     - rebuilds the keys with v_mfma_f32_16x16x32_f16 against the head's
//       up-projection block held in LDS as MFMA fragments (Sec. 3.2, 4.3.3),
//     - rotates them with RoPE at their absolute positions in fp32 (Sec. 3.3),
//     - scores them against the group's query heads with a second MFMA whose
//       k-index is the head dimension (Sec. 3.1).
//   The rows of the score tile are the 16 tokens and the columns are query
//   heads: each KV head only fills its own columns, so up to 16 query heads
//   share one tile.  The online softmax keeps one reference maximum per query
//   head for the whole workgroup (raised only when scores outgrow it), so the
//   probabilities of all waves can be stacked into one matrix and multiplied
//   with the shared value latent V' as one MFMA GEMM, each wave owning a slice
//   of V' channels (the reordered value path of Sec. 3.3 and the stacked
//   p.V' GEMM of App. A.6).  The split's softmax state, value-latent
//   accumulator and the largest approximate scores (rescoring candidates) go
//   to the workspace.
// decode_combine: merges the splits (log-sum-exp weights), rescores the
//   dominant tokens exactly, and applies the value up-projection U_V once per
//   query head (Sec. 3.3), casting to the output type.
#include <hip/hip_runtime.h>

#include <atomic>

#include <type_traits>

#include "starkv_internal.h"

namespace starkv {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2 __attribute__((ext_vector_type(2)));
typedef float f2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f4 mfma16(h8 a, h8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }
__device__ __forceinline__ uint32_t as_u32(h2 h) { return __builtin_bit_cast(uint32_t, h); }

// A pair of 8-bit or 4-bit codes placed in the low mantissa bits of fp16 1024:
// the fp16 value is 1024 + code exactly.  Subtracting 1024 is exact; the fma
// with (s, z) rounds once.
__device__ __forceinline__ uint32_t deq_pair(uint32_t magic_pair, h2 s, h2 z) {
  h2 c = as_h2(magic_pair) - (h2){(_Float16)1024.0f, (_Float16)1024.0f};
  return as_u32(__builtin_elementwise_fma(c, s, z));
}

// Scores may exceed the shared softmax reference by this much (log2 units)
// before it is raised: probabilities stay below 2^8 in fp16.
constexpr float kLazyMargin = 8.0f;

// value-tile precision variants of the split kernel's p.V' phase
constexpr int kValues8 = 0, kValues4 = 1, kValuesMixed = 2;

__device__ __forceinline__ float wave_max16(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}
__device__ __forceinline__ float wave_sum16(float v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}

// ceil(x / k) for 0 <= x < 2^17 + 64 and 1 <= k <= 64, with rk = rcp_up(k),
// the smallest float >= 1/k: the product rounds to the exact quotient's floor
// (x/k is at least 1/64 below the next integer unless it is one, and the
// relative error stays below 2^-22).
__device__ __forceinline__ float rcp_up(int k) {
  float r = __builtin_amdgcn_rcpf((float)k);           // within 1 ulp of 1/k
  const float e = __builtin_fmaf(r, (float)k, -1.0f);  // exact residual
  if (e >= 0.0f) {                                     // step down while still >= 1/k
    const float d = __uint_as_float(__float_as_uint(r) - 1u);
    if (__builtin_fmaf(d, (float)k, -1.0f) >= 0.0f) r = d;
  } else {
    r = __uint_as_float(__float_as_uint(r) + 1u);
  }
  return r;
}
__device__ __forceinline__ int div_up_small(int x, int k, float rk) {
  return (int)((float)(x + k - 1) * rk);
}

// Work plan of one decode step for up to 64 sequences of ragged lengths: the
// split length S = kStepTokens * k is the smallest with at most `cap` work
// items sum_b ceil(L_b / S) (k >= k_lo keeps every sequence at <= 256 splits,
// k <= 64 keeps S <= 8192), and the items are the sequences' splits in order.
// Every wave that calls this gets the same plan.  len: the clamped length held
// by lane b (lanes >= B hold 0).  Returns k; *cnt gets the split count of
// sequence `lane`.
__device__ __forceinline__ int wave_split_plan(int len, int B, int k_lo, int cap, int lane,
                                               int* cnt) {
  const int m = (len + kStepTokens - 1) / kStepTokens;      // steps of sequence `lane`
  const int k = min(k_lo + lane, 64);                       // candidate of this lane
  const float rk = rcp_up(k);
  int items = 0;
  for (int j = 0; j < B; ++j) items += div_up_small(__builtin_amdgcn_readlane(m, j), k, rk);
  const uint64_t ok = __ballot(items <= cap);
  const int ks = ok ? min(k_lo + (int)__builtin_ctzll(ok), 64) : 64;
  *cnt = div_up_small(m, ks, rcp_up(ks));
  return ks;
}

__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}

__device__ __forceinline__ float load_qf(const uint16_t* q, int idx, int bf16) {
  const uint16_t u = q[idx];
  if (bf16) return __uint_as_float(static_cast<uint32_t>(u) << 16);
  return (float)__builtin_bit_cast(_Float16, u);
}

// A value the compiler cannot fold into instructions as a literal, so that it
// stays in a register (lets v_and_or_b32 take it as an operand).
__device__ __forceinline__ uint32_t opaque_u32(uint32_t v) {
  uint32_t r;
  asm volatile("v_mov_b32 %0, %1" : "=v"(r) : "s"(v));
  return r;
}

// 4-bit word of pairs (nibble k, nibble k+4), k = 0..3, with the nibble mask
// held in a register.
__device__ __forceinline__ u4 deq_int4m(uint32_t w, uint32_t mask, h2 s0, h2 z0, h2 s1, h2 z1,
                                        h2 s2, h2 z2, h2 s3, h2 z3) {
  u4 r;
  r.x = deq_pair((w & mask) | 0x64006400u, s0, z0);
  r.y = deq_pair(((w >> 4) & mask) | 0x64006400u, s1, z1);
  r.z = deq_pair(((w >> 8) & mask) | 0x64006400u, s2, z2);
  r.w = deq_pair(((w >> 12) & mask) | 0x64006400u, s3, z3);
  return r;
}

// LDS layout of the split kernel (byte offsets); identical on the host.
struct SplitLds {
  int frag, qc, red, alpha, flag, rot, qmap, loop, raw, vcode, vmeta, pbuf, xch, rope, total;
};

// vcode_bytes: value codes of one step (kStepTokens tokens), a multiple of 16.
__host__ __device__ inline SplitLds split_lds(int frags, int nql, int head_dim, int ct,
                                             int raw_bytes, int v_ng, int vcode_bytes) {
  SplitLds L;
  L.frag = 0;
  L.qc = frags * 1024;
  L.red = L.qc + ((nql * (head_dim + 8) * 2 + 256 + 15) / 16) * 16;
  L.alpha = L.red + kTokenGroups * ct * 16 * 4;
  L.flag = L.alpha + ct * 16 * 4;
  L.rot = L.flag + kWaves * 4;
  L.qmap = L.rot + 64 * 8;
  L.loop = L.qmap + 64 * 4;
  L.raw = L.loop;
  L.vcode = L.raw + kWaves * raw_bytes;
  L.vmeta = L.vcode + vcode_bytes;
  L.pbuf = L.vmeta + 4 * v_ng * 128;
  // single-tile groups of a kernel with one accumulator per half: the second
  // half's partial scores, [token group][lane][8]
  L.xch = L.pbuf + kTokenGroups * ct * 1024;
  int loop_end = L.xch + (ct <= 2 && nql <= 16 ? kTokenGroups * 64 * 32 : 0);
  L.rope = L.vcode;   // RoPE tables (prologue only) alias the value staging
  int rope_end = L.rope + (16 * 65 + 8 * 64) * 8;
  L.total = loop_end > rope_end ? loop_end : rope_end;
  return L;
}

// Asynchronous copy of n_bytes (a multiple of 16) from global memory into LDS by
// the whole workgroup, 16 bytes per lane, without passing through registers.
// Completion is tracked by vmcnt.
__device__ __forceinline__ void copy_to_lds(uint8_t* lds, const uint8_t* src, int n_bytes,
                                            int w, int lane) {
  for (int base = w * 1024; base < n_bytes; base += kWaves * 1024) {
    if (base + lane * 16 < n_bytes)
      __builtin_amdgcn_global_load_lds(src + base + lane * 16, lds + base, 16, 0, 0);
  }
}

// Wait until at most n (wave-uniform) vector memory operations of this wave are
// outstanding; they complete in issue order.  Counts above 15 wait for all
// (conservative).
__device__ __forceinline__ void wait_vm(int n) {
  switch (__builtin_amdgcn_readfirstlane(n)) {
    case 1: __builtin_amdgcn_s_waitcnt(0x0F71); break;
    case 2: __builtin_amdgcn_s_waitcnt(0x0F72); break;
    case 3: __builtin_amdgcn_s_waitcnt(0x0F73); break;
    case 4: __builtin_amdgcn_s_waitcnt(0x0F74); break;
    case 5: __builtin_amdgcn_s_waitcnt(0x0F75); break;
    case 6: __builtin_amdgcn_s_waitcnt(0x0F76); break;
    case 7: __builtin_amdgcn_s_waitcnt(0x0F77); break;
    case 8: __builtin_amdgcn_s_waitcnt(0x0F78); break;
    case 9: __builtin_amdgcn_s_waitcnt(0x0F79); break;
    case 10: __builtin_amdgcn_s_waitcnt(0x0F7A); break;
    case 11: __builtin_amdgcn_s_waitcnt(0x0F7B); break;
    case 12: __builtin_amdgcn_s_waitcnt(0x0F7C); break;
    case 13: __builtin_amdgcn_s_waitcnt(0x0F7D); break;
    case 14: __builtin_amdgcn_s_waitcnt(0x0F7E); break;
    case 15: __builtin_amdgcn_s_waitcnt(0x0F7F); break;
    default: __builtin_amdgcn_s_waitcnt(0x0F70); break;   // vmcnt(0)
  }
}

// Workgroup barrier over LDS traffic only: this wave's LDS operations have
// completed (lgkmcnt(0)), then s_barrier.  The fence of __syncthreads() also
// waits for every global load and LDS copy still in flight (vmcnt(0)); this
// barrier leaves them in flight, and the copies it must cover are waited for
// explicitly (wait_vm) before it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// The same by one wave: n_bytes (a multiple of 16) at src into lds, one copy
// instruction per KiB, lane 0 active in each.
__device__ __forceinline__ void copy_to_lds_wave(uint8_t* lds, const uint8_t* src, int n_bytes,
                                                 int lane) {
  for (int base = 0; base < n_bytes; base += 1024) {
    if (base + lane * 16 < n_bytes)
      __builtin_amdgcn_global_load_lds(src + base + lane * 16, lds + base, 16, 0, 0);
  }
}

__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

// 8-bit codes d (bytes b0..b3) -> fp16 pairs (1024+b0, 1024+b1) and (1024+b2, 1024+b3)
__device__ __forceinline__ u4 deq_int8p(u2 d, h2 s0, h2 z0, h2 s1, h2 z1, h2 s2, h2 z2, h2 s3,
                                        h2 z3) {
  u4 r;
  r.x = deq_pair(perm(0x64646464u, d.x, 0x05010400u), s0, z0);
  r.y = deq_pair(perm(0x64646464u, d.x, 0x05030402u), s1, z1);
  r.z = deq_pair(perm(0x64646464u, d.y, 0x05010400u), s2, z2);
  r.w = deq_pair(perm(0x64646464u, d.y, 0x05030402u), s3, z3);
  return r;
}

// 3-bit codes: the low 24 bits of x hold fields 0..7 (3 bits each).  Fields k
// and k+4 are moved side by side into the two halves of a word and placed in
// the low mantissa bits of fp16 1024 (see deq_pair): pairs (0,4), (1,5), (2,6),
// (3,7).
__device__ __forceinline__ u4 magic_int3(uint32_t x) {
  const uint32_t w2 = (x & 0xFFFu) | ((x << 4) & 0x0FFF0000u);
  u4 m;
  m.x = (w2 & 0x00070007u) | 0x64006400u;
  m.y = ((w2 >> 3) & 0x00070007u) | 0x64006400u;
  m.z = ((w2 >> 6) & 0x00070007u) | 0x64006400u;
  m.w = ((w2 >> 9) & 0x00070007u) | 0x64006400u;
  return m;
}

// Three bytes at LDS byte offset off (any alignment) from two aligned 32-bit
// reads: the code word of a 3-bit lane (and, at a 4-byte aligned offset, the
// whole 32-bit word).
__device__ __forceinline__ uint32_t lds_word_at(const uint8_t* base, int off) {
  const uint32_t* w = reinterpret_cast<const uint32_t*>(base + (off & ~3));
  return __builtin_amdgcn_alignbyte(w[1], w[0], (uint32_t)(off & 3));
}

// Packed fp16 cos/sin of one lane's four RoPE frequencies j0 + e (j0 = 16 kq +
// 4 quad) at one token offset: c01 = (cos j0, cos j0+1), c23, s01, s23.
struct CS4 {
  h2 c01, c23, s01, s23;
};

// 4-bit codes x (nibble k = channel k) -> bytes: nibbles 0,2,4,6 in the first
// word, 1,3,5,7 in the second, so the 8-bit dequantizer applies; the element
// order becomes channels 0,2,4,6,1,3,5,7 (the up-projection fragments match).
__device__ __forceinline__ u2 nibble_bytes(uint32_t x) {
  return (u2){x & 0x0F0F0F0Fu, (x >> 4) & 0x0F0F0F0Fu};
}

// One KV head with KB k-blocks for the wave's 32 tokens: dequantize the key
// latents from the LDS staging area into MFMA operands, rebuild the keys
// (16 rows of the head dimension per MFMA, both halves of every RoPE pair),
// rotate them by the lane's fixed in-step offset (the step's base position is
// applied to the query), and accumulate the scores of the head's query heads.
// The reconstruction of score k-block kbs+1 is issued before the rotation of
// kbs so the matrix cores and the vector ALUs overlap.
// Per-head values used inside the step loop (wave-uniform, read from a lane of
// the wave's head table so that the loop does no scalar memory loads).
struct HeadRt {
  int raw_code, raw_meta, row_bytes, rank, n8, ng8, ngroups, frag_base, gl;
  int64_t code_off, meta_off;
};

template <int D, int QM, int CTH, int KB>
__device__ __forceinline__ void key_head(const HeadRt& kh, const uint8_t* raw, const h8* frag,
                                         const _Float16* qc, int qzero, int gl, int ct0, int G,
                                         int lane, int col, int tcol, int quad,
                                         const CS4 (&cs)[2][D / 32], f4 (&acc_s)[2][CTH]) {
  constexpr int NKBS = D / 32;
  constexpr int QS = D + 8;                  // padded query row (halves)
  const uint8_t* rc = raw + kh.raw_code;
  const uint8_t* rm = raw + kh.raw_meta;
  const int rb16 = 16 * kh.row_bytes;        // bytes of one 16-token block
  // all LDS reads of the head first, then the dequantization.  Lanes whose
  // chunk lies beyond the rank read chunk 0 (finite values that meet zero
  // up-projection rows).
  u2 code[2][KB];
  uint32_t meta[2][KB];
  u4 cf[2][KB];
  bool is8[KB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
    const int c = 4 * kb + quad;
    const bool valid = (kb < KB - 1) || (8 * c < kh.rank);
    if (QM == STARKV_Q_F16) {
      const int off = valid ? kb * 1024 + quad * 256 + tcol * 16 : 0;
#pragma unroll
      for (int s = 0; s < 2; ++s) cf[s][kb] = *reinterpret_cast<const u4*>(rc + s * rb16 + off);
    } else if (QM == STARKV_Q_MIX4_3) {
      // outlier chunks (4-bit, 64 B per 16 tokens) first, then 3-bit chunks (48 B)
      is8[kb] = c < kh.n8;
      int off = is8[kb] ? kb * 256 + quad * 64 + tcol * 4 : kh.n8 * 64 + (c - kh.n8) * 48 + tcol * 3;
      int gi = is8[kb] ? c / 4 : kh.ng8 + (c - kh.n8) / 4;
      if (!valid) { off = 0; gi = 0; }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        meta[s][kb] = *reinterpret_cast<const uint32_t*>(rm + (s * kh.ngroups + gi) * 64 + tcol * 4);
        code[s][kb].x = lds_word_at(rc + s * rb16, off);
      }
    } else {
      is8[kb] = QM == STARKV_Q_MIX8_4 && c < kh.n8;
      int off = is8[kb] ? kb * 512 + quad * 128 + tcol * 8 : kh.n8 * 64 + kb * 256 + quad * 64 + tcol * 4;
      int gi = is8[kb] ? c / 4 : kh.ng8 + (c - kh.n8) / 4;
      if (!valid) { off = 0; gi = 0; }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        meta[s][kb] = *reinterpret_cast<const uint32_t*>(rm + (s * kh.ngroups + gi) * 64 + tcol * 4);
        if (QM == STARKV_Q_INT4) {
          code[s][kb].x = *reinterpret_cast<const uint32_t*>(rc + s * rb16 + off);
        } else {
          // 8-byte aligned reads only (a 4-bit lane takes its half of the word)
          const u2 d = *reinterpret_cast<const u2*>(rc + s * rb16 + (off & ~7));
          code[s][kb] = d;
          if (off & 4) code[s][kb].x = d.y;
        }
      }
    }
  }
  h8 xop[2][KB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      u4 v;
      if (QM == STARKV_Q_F16) {
        v = cf[s][kb];
      } else {
        const uint32_t mz = meta[s][kb];
        const h2 sv = as_h2(perm(mz, mz, 0x01000100u));
        const h2 zv = as_h2(perm(mz, mz, 0x03020302u));
        u2 d = code[s][kb];
        const u2 nb = nibble_bytes(d.x);
        if (QM == STARKV_Q_MIX4_3) {
          // 4-bit lanes: nibble bytes; 3-bit lanes: field pairs (element orders
          // 0,2,4,6,1,3,5,7 and 0,4,1,5,2,6,3,7; the fragments match)
          const u4 m3 = magic_int3(d.x);
          u4 m;
          m.x = is8[kb] ? perm(0x64646464u, nb.x, 0x05010400u) : m3.x;
          m.y = is8[kb] ? perm(0x64646464u, nb.x, 0x05030402u) : m3.y;
          m.z = is8[kb] ? perm(0x64646464u, nb.y, 0x05010400u) : m3.z;
          m.w = is8[kb] ? perm(0x64646464u, nb.y, 0x05030402u) : m3.w;
          v = (u4){deq_pair(m.x, sv, zv), deq_pair(m.y, sv, zv), deq_pair(m.z, sv, zv),
                   deq_pair(m.w, sv, zv)};
        } else {
          if (QM == STARKV_Q_INT4) {
            d = nb;
          } else {
            d.x = is8[kb] ? d.x : nb.x;
            d.y = is8[kb] ? d.y : nb.y;
          }
          v = deq_int8p(d, sv, zv, sv, zv, sv, zv, sv, zv);
        }
      }
      xop[s][kb] = __builtin_bit_cast(h8, v);
    }
  }
  const int ct_g = (gl * G) / 16 - ct0;      // score tile of this head within the half
  const int c_lo = (gl * G) % 16;
  const bool mine = col >= c_lo && col < c_lo + G;
  // the lane's query vectors of k-blocks 0.. are 32 halves apart; lanes whose
  // column is not one of the head's queries read a zero area laid out alike
  const _Float16* qb = qc + (mine ? (((gl * G) / 16) * 16 + col) * QS : qzero) + quad * 8;
  const int fb = kh.frag_base;
  f4 klo[2][2], khi[2][2];   // [buffer][subtile]
#pragma unroll
  for (int kbs = 0; kbs <= NKBS; ++kbs) {
    if (kbs < NKBS) {        // reconstruct rows 16*kbs.. and 16*kbs + D/2..
      const int bufn = kbs & 1;
#pragma unroll
      for (int s = 0; s < 2; ++s) { klo[bufn][s] = (f4){0, 0, 0, 0}; khi[bufn][s] = (f4){0, 0, 0, 0}; }
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const h8 a_lo = frag[(fb + kbs * KB + kb) * 64 + lane];
        const h8 a_hi = frag[(fb + (kbs + NKBS) * KB + kb) * 64 + lane];
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          klo[bufn][s] = mfma16(a_lo, xop[s][kb], klo[bufn][s]);
          khi[bufn][s] = mfma16(a_hi, xop[s][kb], khi[bufn][s]);
        }
      }
    }
    if (kbs > 0) {           // rotate and score k-block kbs-1 (packed fp16)
      const int kq = kbs - 1, buf = kq & 1;
      const h8 qf = *reinterpret_cast<const h8*>(qb + kq * 32);
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const CS4& r = cs[s][kq];
        const f4 a = klo[buf][s], bb = khi[buf][s];
        const h2 a01 = __builtin_convertvector((f2){a[0], a[1]}, h2);
        const h2 a23 = __builtin_convertvector((f2){a[2], a[3]}, h2);
        const h2 b01 = __builtin_convertvector((f2){bb[0], bb[1]}, h2);
        const h2 b23 = __builtin_convertvector((f2){bb[2], bb[3]}, h2);
        u4 kr;
        kr[0] = as_u32(__builtin_elementwise_fma(a01, r.c01, -(b01 * r.s01)));
        kr[1] = as_u32(__builtin_elementwise_fma(a23, r.c23, -(b23 * r.s23)));
        kr[2] = as_u32(__builtin_elementwise_fma(b01, r.c01, a01 * r.s01));
        kr[3] = as_u32(__builtin_elementwise_fma(b23, r.c23, a23 * r.s23));
        const h8 kop = __builtin_bit_cast(h8, kr);
#pragma unroll
        for (int c = 0; c < CTH; ++c)
          if (CTH == 1 || c == ct_g) acc_s[s][c] = mfma16(kop, qf, acc_s[s][c]);
      }
    }
  }
}

// Dequantize a pair of codes placed in the low mantissa bits of fp16 1024 (see
// deq_pair) with the (scale, zero) pair packed in one word: the scale and the
// zero reach both halves of the fma through its operand selects.
__device__ __forceinline__ uint32_t deq_pair_mz(uint32_t magic_pair, uint32_t mz) {
  const h2 c = as_h2(magic_pair) - (h2){(_Float16)1024.0f, (_Float16)1024.0f};
  const h2 m = as_h2(mz);
  return as_u32(__builtin_elementwise_fma(c, __builtin_shufflevector(m, m, 0, 0),
                                          __builtin_shufflevector(m, m, 1, 1)));
}

// The last score k-block of a head, rebuilt but not yet rotated and scored: the
// next head finishes it after issuing its own LDS reads, so that this work
// covers their latency and the next head's first matrix work (key_head_q).
template <int CTH>
struct KeyPending {
  f4 lo[2], hi[2];   // reconstructed rows 16*kq.. and 16*kq + D/2.. per subtile
  h8 q;              // query operand of that k-block
  int ct;            // score tile of the head within the half
};

// Rotate one k-block of rebuilt keys (rows j and j + D/2 of the lane's token, in
// fp32) by the lane's fixed RoPE rotation, in packed fp16, and accumulate the
// scores of the head's query columns.
template <int CTH>
__device__ __forceinline__ void rotate_score(const f4& a, const f4& bb, const CS4& r, const h8& qf,
                                             int ct, f4 (&acc)[CTH]) {
  const h2 a01 = __builtin_convertvector((f2){a[0], a[1]}, h2);
  const h2 a23 = __builtin_convertvector((f2){a[2], a[3]}, h2);
  const h2 b01 = __builtin_convertvector((f2){bb[0], bb[1]}, h2);
  const h2 b23 = __builtin_convertvector((f2){bb[2], bb[3]}, h2);
  u4 kr;
  kr[0] = as_u32(__builtin_elementwise_fma(a01, r.c01, -(b01 * r.s01)));
  kr[1] = as_u32(__builtin_elementwise_fma(a23, r.c23, -(b23 * r.s23)));
  kr[2] = as_u32(__builtin_elementwise_fma(b01, r.c01, a01 * r.s01));
  kr[3] = as_u32(__builtin_elementwise_fma(b23, r.c23, a23 * r.s23));
  const h8 kop = __builtin_bit_cast(h8, kr);
#pragma unroll
  for (int c = 0; c < CTH; ++c)
    if (CTH == 1 || c == ct) acc[c] = mfma16(kop, qf, acc[c]);
}

template <int D, int CTH>
__device__ __forceinline__ void key_drain(const KeyPending<CTH>& pd, const CS4 (&cs)[2][D / 32],
                                          f4 (&acc_s)[2][CTH]) {
#pragma unroll
  for (int s = 0; s < 2; ++s) rotate_score<CTH>(pd.lo[s], pd.hi[s], cs[s][D / 32 - 1], pd.q, pd.ct, acc_s[s]);
}

// key_head for the 4-bit and the 8-bit/4-bit caches.  In these formats a head
// with KB k-blocks has exactly KB 8-bit chunks (8 * ceil(r / 32) outlier
// channels) or none, so only k-block 0 mixes the two widths (lanes of chunk quad
// < KB read 8 bytes, the others 4), and every LDS offset is a per-lane constant
// plus a compile-time part: lc4 = 64 quad + 4 tcol (4-bit chunk layout), lc8 =
// 128 quad + 8 tcol (8-bit).  A lane reads two words of k-block 0 (8-bit lanes
// the two words of their 8 codes, 4-bit lanes the same word twice) and spreads
// them into bytes with a per-lane shift and mask, so both widths run the same
// instructions.  The head runs as a pipeline over its score k-blocks: the
// matrix cores rebuild k-block kbs while the rotation and scores of kbs - 1 run
// on the vector ALUs, the fragments of kbs + 1 and the query operand of kbs are
// read one stage ahead, and the last k-block is left pending for the next head
// (or the caller's drain).
template <int D, int QM, int CTH, int KB>
__device__ __forceinline__ void key_head_q(const HeadRt& kh, const uint8_t* raw, const h8* frag,
                                           const _Float16* qc, int qzero, int gl, int ct0, int G,
                                           int lane, int col, int tcol, int quad, int lc4, int lc8,
                                           const CS4 (&cs)[2][D / 32], f4 (&acc_s)[2][CTH],
                                           KeyPending<CTH>& pend) {
  constexpr bool MIX = QM == STARKV_Q_MIX8_4;
  constexpr int NKBS = D / 32;
  constexpr int QS = D + 8;
  constexpr int X4 = MIX ? 64 * KB : 0;      // first 4-bit chunk of a 16-token block
  const bool is8 = MIX && quad < KB;          // k-block 0 chunk of this lane is 8-bit
  const int rb16 = 16 * kh.row_bytes;         // bytes of one 16-token block
  const int mg64 = 64 * kh.ngroups;           // meta bytes of one 16-token block
  const uint8_t* rc = raw + kh.raw_code;
  // group of chunk 4 kb + quad: kb + 1 for the 4-bit chunks of a mixed head, kb otherwise
  const uint8_t* rm = raw + kh.raw_meta + 4 * tcol + ((MIX && quad >= KB) ? 64 : 0);
  // Lanes whose chunk of the last k-block lies beyond the rank read the codes and
  // group 0's meta of chunk 0 instead: finite values that meet zero fragment rows.
  const bool vlast = 8 * (4 * (KB - 1) + quad) < kh.rank;
  const uint8_t* rm0 = raw + kh.raw_meta + 4 * tcol;
  const uint8_t* rml = vlast ? rm : rm0;
  const int a0 = (KB > 1 || vlast) ? (is8 ? lc8 : lc4 + X4) : 8 * tcol;
  const int a0b = (KB > 1 || vlast) ? (is8 ? lc8 + 4 : lc4 + X4) : 8 * tcol;
  const int alast = vlast ? lc4 + X4 + 256 * (KB - 1) : 8 * tcol;
  const uint32_t mk0 = is8 ? 0xFFFFFFFFu : 0x0F0F0F0Fu;
  const uint32_t sh0 = is8 ? 0u : 4u;
  const int ct_g = (gl * G) / 16 - ct0;      // score tile of this head within the half
  const int c_lo = (gl * G) % 16;
  const bool mine = col >= c_lo && col < c_lo + G;
  const _Float16* qb = qc + (mine ? (((gl * G) / 16) * 16 + col) * QS : qzero) + quad * 8;
  const h8* fr = frag + kh.frag_base * 64 + lane;
  // the codes and meta of this head's tokens
  uint32_t w0[2], w1[2], wk[2][KB], mz[2][KB];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      if (kb == 0) {
        w0[s] = *reinterpret_cast<const uint32_t*>(rc + s * rb16 + a0);
        w1[s] = *reinterpret_cast<const uint32_t*>(rc + s * rb16 + a0b);
      } else {
        const int a = kb == KB - 1 ? alast : lc4 + X4 + 256 * kb;
        wk[s][kb] = *reinterpret_cast<const uint32_t*>(rc + s * rb16 + a);
      }
      mz[s][kb] = kb == KB - 1
          ? *reinterpret_cast<const uint32_t*>(rml + s * mg64 + (vlast ? 64 * kb : 0))
          : *reinterpret_cast<const uint32_t*>(rm + s * mg64 + 64 * kb);
    }
  }
  // heads of up to two k-blocks read the next stage's fragments one stage ahead
  // (two buffers); larger ones read a stage's fragments at its start.  The
  // query operand of a stage is read one stage ahead.
  constexpr bool kAhead = KB <= 2;
  h8 alo[KB], ahi[KB];
  if (kAhead) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      alo[kb] = fr[kb * 64];
      ahi[kb] = fr[(NKBS * KB + kb) * 64];
    }
  }
  h8 qcur = *reinterpret_cast<const h8*>(qb);
  __builtin_amdgcn_sched_barrier(0);
  // the previous head's last k-block while these reads are in flight
  key_drain<D, CTH>(pend, cs, acc_s);
  __builtin_amdgcn_sched_barrier(0);
  h8 xop[2][KB];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      uint32_t lo, hi;
      if (kb == 0) {
        lo = w0[s] & mk0;
        hi = (w1[s] >> sh0) & mk0;
      } else {
        lo = wk[s][kb] & 0x0F0F0F0Fu;
        hi = (wk[s][kb] >> 4) & 0x0F0F0F0Fu;
      }
      u4 v;
      v.x = deq_pair_mz(perm(0x64646464u, lo, 0x05010400u), mz[s][kb]);
      v.y = deq_pair_mz(perm(0x64646464u, lo, 0x05030402u), mz[s][kb]);
      v.z = deq_pair_mz(perm(0x64646464u, hi, 0x05010400u), mz[s][kb]);
      v.w = deq_pair_mz(perm(0x64646464u, hi, 0x05030402u), mz[s][kb]);
      xop[s][kb] = __builtin_bit_cast(h8, v);
    }
  }
  f4 klo[2][2], khi[2][2];   // [buffer][subtile]
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int kbs = 0; kbs < NKBS; ++kbs) {
    h8 nlo[KB], nhi[KB], qnext;
    if (kbs > 0) qnext = *reinterpret_cast<const h8*>(qb + kbs * 32);
    const int ks = kAhead ? kbs + 1 : kbs;   // stage whose fragments are read now
    if (ks < NKBS) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        nlo[kb] = fr[(ks * KB + kb) * 64];
        nhi[kb] = fr[((ks + NKBS) * KB + kb) * 64];
      }
    }
    if (!kAhead) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        alo[kb] = nlo[kb];
        ahi[kb] = nhi[kb];
      }
    }
    // keep the fragment reads ahead of this stage's matrix work
    __builtin_amdgcn_sched_barrier(0);
    {                        // reconstruct rows 16*kbs.. and 16*kbs + D/2..
      const int bufn = kbs & 1;
#pragma unroll
      for (int s = 0; s < 2; ++s) { klo[bufn][s] = (f4){0, 0, 0, 0}; khi[bufn][s] = (f4){0, 0, 0, 0}; }
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          klo[bufn][s] = mfma16(alo[kb], xop[s][kb], klo[bufn][s]);
          khi[bufn][s] = mfma16(ahi[kb], xop[s][kb], khi[bufn][s]);
          // in this order, first: left to itself the scheduler sinks them to the
          // end of the stage, where the next stage's rotation waits on them
          __builtin_amdgcn_sched_barrier(0);
        }
    }
    if (kbs > 0) {           // rotate and score k-block kbs-1
      const int kq = kbs - 1, buf = kq & 1;
#pragma unroll
      for (int s = 0; s < 2; ++s) rotate_score<CTH>(klo[buf][s], khi[buf][s], cs[s][kq], qcur, ct_g, acc_s[s]);
    }
    if (kAhead && kbs + 1 < NKBS) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        alo[kb] = nlo[kb];
        ahi[kb] = nhi[kb];
      }
    }
    if (kbs > 0) qcur = qnext;
    __builtin_amdgcn_sched_barrier(0);
  }
  // the last k-block waits for the next head (or the caller's drain)
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    pend.lo[s] = klo[(NKBS - 1) & 1][s];
    pend.hi[s] = khi[(NKBS - 1) & 1][s];
  }
  pend.q = qcur;
  pend.ct = ct_g;
}

// The group's query heads rotated to the step's base position t (RoPE applied to
// the query as R(t)^T q, so that q . R(t + u) k = (R(t)^T q) . (R(u) k)), one
// padded fp16 row per head, permuted so that lane (col, quad) of score k-block
// kbs reads one 16-byte vector: elements e = q'[j0 + e], 4 + e = q'[j0 + e + D/2],
// j0 = 16*kbs + 4*quad.  Thread t owns vectors t, t + 512, .. (frequencies
// j0 .. j0+3 fixed per thread).
template <int D, int NQV>
__device__ __forceinline__ void store_rotated_q(_Float16* qc, int nql, int tid,
                                                const float (&qo)[NQV][8], const float2 (&bs)[4]) {
  // qo holds the query already multiplied by log2(e)/sqrt(d)
  constexpr int QS = D + 8;
  constexpr int NV = D / 8;                  // vectors per query row
#pragma unroll
  for (int v = 0; v < NQV; ++v) {
    const int vi = tid + v * kThreads;
    const int il = vi / NV, jg = vi % NV;
    if (il < nql) {
      u4 o;
#pragma unroll
      for (int e = 0; e < 4; e += 2) {
        float lo[2], hi[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const float a = qo[v][e + u], b = qo[v][4 + e + u];
          const float c = bs[e + u].x, s = bs[e + u].y;
          lo[u] = __builtin_fmaf(a, c, b * s);
          hi[u] = __builtin_fmaf(b, c, -(a * s));
        }
        o[e / 2] = as_u32(__builtin_convertvector((f2){lo[0], lo[1]}, h2));
        o[2 + e / 2] = as_u32(__builtin_convertvector((f2){hi[0], hi[1]}, h2));
      }
      *reinterpret_cast<u4*>(qc + il * QS + jg * 8) = o;
    }
  }
}

// CT: score tiles (16 query heads) of a head group; CTH = tiles of one half;
// NTW: value-channel tiles (16 channels) per wave.
template <int D, int QM, int CT, int NTW>
__global__ __launch_bounds__(kThreads, 1) void decode_split_kernel(DecodeParams p) {
  extern __shared__ __align__(16) uint8_t smem[];
  constexpr int CTH = (CT + 1) / 2;
  constexpr int NKBS = D / 32;   // score k-blocks (head dimension / 32)
  // The pipelined key routine (key_head_q) for the 4-bit and 8-bit/4-bit caches
  // when the value accumulators are small (NTW <= 2): with more, its state
  // across heads no longer fits in registers and key_head is faster.
  constexpr bool kPipeKeys = (QM == STARKV_Q_INT4 || QM == STARKV_Q_MIX8_4) && NTW <= 2;
  // alternate issue priority between the two waves of a SIMD (key phase);
  // measured faster with up to two value tiles per wave, slower with four
  constexpr bool kAltPrio = NTW <= 2;
  constexpr int HALF = D / 2;
  constexpr int QS = D + 8;
  constexpr int NQV = (16 * CT * (D / 8) + kThreads - 1) / kThreads;   // query vectors per thread
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Waves w and w + 4 share a SIMD and take the two halves of the heads on the
  // same tokens, so every SIMD carries the whole key work of one token group
  // (the halves cannot always be balanced: ranks 80, 32, 128, 128 split 9 : 11
  // in k-block cost).
  const int tg = w & (kTokenGroups - 1);   // token group: tokens 32*tg.. of each step
  const int hh = w / kTokenGroups;         // half of the group's KV heads
  const int col = lane & 15, quad = lane >> 4;
  // Token order of the score tiles: row 4*quad + e of a 16-token subtile is
  // token 4*e + quad, so a lane's rows are tokens quad, quad+4, quad+8,
  // quad+12 -- consecutive tokens (an attention sink, a local cluster) fall in
  // different lanes and so in different rescoring candidates.  The key
  // reconstruction reads token tcol into MFMA column col, and the value chunks
  // hold their slots in the same order.
  const int tcol = 4 * (col & 3) + (col >> 2);
  // LDS offsets of this lane's key codes inside a 16-token block (4-bit and 8-bit chunk layouts)
  const int lc4 = 64 * quad + 4 * tcol, lc8 = 128 * quad + 8 * tcol;
  const int hg = blockIdx.z;
  const int g0 = p.hg_first[hg], g1 = p.hg_first[hg + 1], gm = p.hg_mid[hg];
  const int G = p.group_q;
  const int nql = (g1 - g0) * G;
  const int ct_half = ((gm - g0) * G + 15) / 16;          // score tiles of the first half
  // A single-tile group (one accumulator per half: CT <= 2) splits its heads
  // between the halves by key cost; the first half owns the tile and adds the
  // second half's partial scores to its own before the softmax.
  const bool merge = CTH == 1 && nql <= 16 && g1 > gm;
  const int ct0 = hh ? ct_half : 0;                        // first score tile of this half
  const int ctn = hh ? (nql + 15) / 16 - ct_half : ct_half; // its tile count

  // ---------------------------------------------------------------- prologue
  // Every load whose address is known at entry is issued first (context
  // length, this half's head table, the fragment table, the query heads of
  // this thread's query vectors); the key copies of step 0, the fragment and
  // query loads follow, and the RoPE tables are computed while they are in
  // flight.  The prologue then costs about two memory round trips.
  // context length: of this workgroup's sequence, or (work plan over ragged
  // lengths) of sequence `lane`
  int L = p.dyn ? (lane < p.batch ? p.ctx_len[lane] : 0) : p.ctx_len[blockIdx.y];
  // The half's heads in processing order (grouped by k-block count): lane i
  // of the head table holds the i-th head's packed fields (staging offsets;
  // row bytes, rank, 8-bit chunks, 8-bit groups, groups, slot; fragment base;
  // plane offsets / 256).
  const int c0 = p.cls[hg][hh][0];
  int cls_end[NKBS + 1];
#pragma unroll
  for (int k = 0; k <= NKBS; ++k) cls_end[k] = p.cls[hg][hh][k] - c0;
  const int n_h = cls_end[NKBS];
  uint32_t t_raw = 0, t_geo = 0, t_fb = 0, t_code = 0, t_meta = 0;
  if (lane < n_h) {
    t_raw = p.o_raw[c0 + lane];
    t_geo = p.o_geo[c0 + lane];
    t_fb = p.o_fb[c0 + lane];
    t_code = p.o_code[c0 + lane];
    t_meta = p.o_meta[c0 + lane];
  }
  // fragment table: lane i holds slot g0 + i (first fragment, k-blocks,
  // 8-bit chunks, rank, first B_k row)
  int l_fb = 0x7FFFFFFF, l_nkb = 1, l_n8 = 0, l_rank = 1, l_row = 0;
  if (lane < g1 - g0) {
    const KHeadInfo& k = p.kh[g0 + lane];
    l_fb = k.frag_base;
    l_nkb = k.nkb;
    l_n8 = k.n8;
    l_rank = k.rank;
    l_row = k.bk_row;
  }
  // query head of each of this thread's query vectors
  int qh[NQV];
#pragma unroll
  for (int v = 0; v < NQV; ++v) {
    const int il = (tid + v * kThreads) / (D / 8);
    qh[v] = il < nql ? p.kh[g0 + il / G].head * G + il % G : 0;
  }
  const int qm = tid < nql ? p.kh[g0 + tid / G].head * G + tid % G : 0;
  L = L < 0 ? 0 : (L > p.max_ctx ? p.max_ctx : L);
  // the work item: sequence b, its split, the split length S, and the slot of
  // the item's partials
  int b, split, S, pitem;
  if (p.dyn) {
    int cnt;
    S = wave_split_plan(L, p.batch, p.k_lo, p.cap, lane, &cnt) * kStepTokens;
    if (blockIdx.x == 0 && blockIdx.z == 0 && w == 0) {
      // the plan of every sequence for the merge pass: its first item (an
      // exclusive prefix sum of the split counts), split count and length
      int incl = lane < p.batch ? cnt : 0;
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
      }
      if (lane < p.batch)
        *reinterpret_cast<int4*>(p.plan + 4 * lane) = make_int4(incl - cnt, cnt, L, 0);
    }
    pitem = blockIdx.x;
    // the item's sequence: a scalar walk over the sequences' split counts
    b = -1;
    split = pitem;
    for (int j = 0; j < p.batch; ++j) {
      const int cj = __builtin_amdgcn_readlane(cnt, j);
      if (split < cj) { b = j; break; }
      split -= cj;
    }
    if (b < 0) return;                      // past the last item
    L = __builtin_amdgcn_readlane(L, b);
  } else {
    b = blockIdx.y;
    split = blockIdx.x;
    S = p.split_len;
    pitem = b * p.n_split + split;
  }
  const int t_begin = split * S;
  if (t_begin >= L) return;
  const int t_end = min(t_begin + S, L);
  // Paged caches: lane j holds the pool page of the split's j-th page (a split
  // of at most 8192 tokens spans at most 64 pages of at least 128 tokens).
  const int pg_first = p.rmap.table ? t_begin >> p.rmap.shift : 0;
  int l_page = 0;
  if (p.rmap.table) {
    const int pj = min(pg_first + lane, p.rmap.per_seq - 1);
    const int pg = p.rmap.table[(int64_t)b * p.rmap.per_seq + pj];
    l_page = pg < 0 ? 0 : (pg >= p.rmap.n_pages ? p.rmap.n_pages - 1 : pg);
  }
  const int n_steps = (t_end - t_begin + kStepTokens - 1) / kStepTokens;

  const int raw_bytes = p.hg_raw_bytes[hg];
  const int vcode_bytes = kStepTokens * p.v_row_bytes;
  const SplitLds LL = split_lds(p.hg_frags[hg], nql, D, CT, raw_bytes, p.v_ng, vcode_bytes);
  h8* frag = reinterpret_cast<h8*>(smem + LL.frag);
  _Float16* qc = reinterpret_cast<_Float16*>(smem + LL.qc);
  float* red = reinterpret_cast<float*>(smem + LL.red);
  float* alpha_s = reinterpret_cast<float*>(smem + LL.alpha);
  int* flag_s = reinterpret_cast<int*>(smem + LL.flag);
  float2* rot_s = reinterpret_cast<float2*>(smem + LL.rot);        // [64] step rotations
  int* qmap = reinterpret_cast<int*>(smem + LL.qmap);             // slot-local -> query head
  uint8_t* raw = smem + LL.raw + w * raw_bytes;
  uint8_t* vcode = smem + LL.vcode;
  uint8_t* vmeta = smem + LL.vmeta;
  h8* pbuf = reinterpret_cast<h8*>(smem + LL.pbuf);
  float2* rope_col = reinterpret_cast<float2*>(smem + LL.rope);   // [16][65]
  float2* rope_ws = rope_col + 16 * 65;   // [8][64]; rope_col rows are padded to 65 (banks)
  const int qzero = nql * QS;

  if (tid < nql) qmap[tid] = qm;
  if (tid < 128) qc[qzero + tid] = (_Float16)0.0f;
  // Key staging: the wave's 32 tokens of every key head of its half, codes then
  // meta per head, copied straight into the wave's LDS area.  A head's copy for
  // the next step is issued as soon as the head has been processed, so the
  // copies have most of a step to land.  Lane 0 of every issued copy is active,
  // so the wave issues exactly n_kw copies per step.
  // cache row of the first token of a step (steps never cross a page)
  auto step_row = [&](int step) -> int64_t {
    const int t = t_begin + step * kStepTokens;
    if (!p.rmap.table) return (int64_t)b * p.rmap.cap_pad + t;
    const int pg = __builtin_amdgcn_readlane(l_page, min((t >> p.rmap.shift) - pg_first, 63));
    return ((int64_t)pg << p.rmap.shift) + (t & ((1 << p.rmap.shift) - 1));
  };
  // blk: the wave's first 16-token key block of the step
  auto copy_head = [&](const HeadRt& kh, int64_t blk) {
    copy_to_lds_wave(raw + kh.raw_code, p.cache + kh.code_off + blk * 16 * kh.row_bytes,
                     32 * kh.row_bytes, lane);
    if (QM != STARKV_Q_F16)
      copy_to_lds_wave(raw + kh.raw_meta, p.cache + kh.meta_off + blk * kh.ngroups * 64,
                       2 * kh.ngroups * 64, lane);
  };
  auto head_rt = [&](int i) {
    HeadRt h;
    const uint32_t raw_ = __builtin_amdgcn_readlane(t_raw, i);
    const uint32_t geo = __builtin_amdgcn_readlane(t_geo, i);
    h.raw_code = (int)(raw_ & 0xFFFFu);
    h.raw_meta = (int)(raw_ >> 16);
    h.row_bytes = (int)(geo & 0x1FFu);
    h.rank = (int)((geo >> 9) & 0xFFu);
    h.n8 = (int)((geo >> 17) & 7u);
    h.ng8 = (int)((geo >> 20) & 3u);
    h.ngroups = (int)((geo >> 22) & 7u);
    h.gl = (int)((geo >> 25) & 15u);
    h.frag_base = (int)__builtin_amdgcn_readlane(t_fb, i);
    h.code_off = (int64_t)__builtin_amdgcn_readlane(t_code, i) << 8;
    h.meta_off = (int64_t)__builtin_amdgcn_readlane(t_meta, i) << 8;
    return h;
  };
  int n_kw = 0;   // key copies per step
  {
    int l_kw = 0;
    if (lane < n_h) {
      const int rb = (int)(t_geo & 0x1FFu), ng = (int)((t_geo >> 22) & 7u);
      l_kw = (32 * rb + 1023) / 1024;
      if (QM != STARKV_Q_F16) l_kw += (2 * ng * 64 + 1023) / 1024;
    }
    for (int i = 0; i < n_h; ++i) n_kw += __builtin_amdgcn_readlane(l_kw, i);
  }
  // step 0's key copies (the key staging is not used by the prologue)
  {
    const int64_t blk0 = (step_row(0) + 32 * tg) >> 4;
    for (int i = 0; i < n_h; ++i) copy_head(head_rt(i), blk0);
  }

  // Up-projection fragments.  Fragment (slot, m-tile mt, k-block kb), lane
  // (jj, kq): 8 halves = B_k[row][16*mt + jj] for the 8 channels of chunk
  // 4*kb + kq, in the order the key operand delivers them (4-bit chunks:
  // channels 0,2,4,6,1,3,5,7; 8-bit and fp16 chunks in order); channels at or
  // beyond the rank are zero.  Wave w builds fragments w, w + 8, ... in batches
  // whose loads are all issued first.  A fragment's 32 x 16 block of B_k
  // arrives as one 16-byte load per lane (block row l/2, columns 8*(l%2)..),
  // is written row-major into the fragment's own 1 KiB of LDS, and is read
  // back in operand order by the same wave, whose LDS operations complete in
  // issue order.
  constexpr int kBatch = 5;
  const int n_fr = p.hg_frags[hg];
  // rows beyond the rank (and fragments beyond the group) load a valid row and
  // are zeroed when stored, so no load sits behind a branch; info = row live
  // (bit 0) | element order of the chunk this lane reads back (bits 1..)
  auto frag_load = [&](int f0, u4 (&ld)[kBatch], uint32_t (&info)[kBatch]) {
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int f = min(f0 + k * kWaves, n_fr - 1);
      // the fragment's slot: the last one whose first fragment is <= f
      const int hs = __builtin_popcountll(__ballot(l_fb <= f)) - 1;
      const int fb = __builtin_amdgcn_readlane(l_fb, hs);
      const int nkb = __builtin_amdgcn_readlane(l_nkb, hs);
      const int n8 = __builtin_amdgcn_readlane(l_n8, hs);
      const int rank = __builtin_amdgcn_readlane(l_rank, hs);
      const int bk_row = __builtin_amdgcn_readlane(l_row, hs);
      const int fl = f - fb;
      const int mt = fl / nkb, kb = fl % nkb;
      const int row = 32 * kb + (lane >> 1);
      ld[k] = *reinterpret_cast<const u4*>(p.bk + (int64_t)(bk_row + min(row, rank - 1)) * D +
                                           16 * mt + 8 * (lane & 1));
      // element order of the chunk's key operand: 8-bit and fp16 in order,
      // 4-bit 0,2,4,6,1,3,5,7, 3-bit 0,4,1,5,2,6,3,7
      const int c = 4 * kb + (lane >> 4);
      const int ord = QM == STARKV_Q_F16 ? 0
                      : QM == STARKV_Q_MIX4_3 ? (c < n8 ? 1 : 2) : (c < n8 ? 0 : 1);
      info[k] = (row < rank ? 1u : 0u) | ((uint32_t)ord << 1);
    }
  };
  auto wave_sync = [] {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };
  auto frag_store = [&](int f0, const u4 (&ld)[kBatch], const uint32_t (&info)[kBatch]) {
    const int jj = lane & 15, kq = lane >> 4;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int f = f0 + k * kWaves;          // wave-uniform
      if (f < n_fr) {
        u4* slot = reinterpret_cast<u4*>(frag + f * 64);
        slot[lane] = (info[k] & 1u) ? ld[k] : (u4){0, 0, 0, 0};
        wave_sync();
        const uint16_t* blk = reinterpret_cast<const uint16_t*>(slot);   // [32][16]
        const int ord = (int)(info[k] >> 1);
        uint32_t e8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int wi = ord == 0 ? e : ord == 1 ? (e < 4 ? 2 * e : 2 * (e - 4) + 1)
                                                 : (e % 2 == 0 ? e / 2 : 4 + e / 2);
          e8[e] = blk[(8 * kq + wi) * 16 + jj];
        }
        wave_sync();
        u4 v;
#pragma unroll
        for (int h = 0; h < 4; ++h) v[h] = e8[2 * h] | (e8[2 * h + 1] << 16);
        slot[lane] = v;
      }
    }
  };
  // the fragment area is free from the start: batch 0 is loaded here and
  // stored after the RoPE tables are computed, batch 1 is loaded then and
  // stored after the key rotations, and any further batches follow
  u4 ld0[kBatch], ld1[kBatch];
  uint32_t live0[kBatch], live1[kBatch];
  frag_load(w, ld0, live0);

  // this thread's query vectors (fp32) and the base rotation of its four
  // frequencies at t_begin (angle reduced in fp64)
  float qo[NQV][8];
  float2 bs[4];
  {
    const int jg = tid % (D / 8);
    const int j0 = 4 * jg;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const double om = exp2(-(2.0 * (j0 + e) / D) * p.log2_theta);
      double a = (double)t_begin * om;
      a -= 6.283185307179586476925286766559 * floor(a * 0.15915494309189533576888376337251);
      double sa, ca;
      sincos(a, &sa, &ca);
      bs[e] = make_float2((float)ca, (float)sa);
    }
#pragma unroll
    for (int v = 0; v < NQV; ++v) {
      const uint16_t* qs = static_cast<const uint16_t*>(p.q) + ((int64_t)b * p.n_q + qh[v]) * D;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        qo[v][e] = load_qf(qs, j0 + e, p.q_bf16) * p.score_scale;
        qo[v][4 + e] = load_qf(qs, j0 + e + HALF, p.q_bf16) * p.score_scale;
      }
    }
  }
  // RoPE tables: the lane's in-step offset u = 32*tg + 16*s + col composed as
  // the subtile rotation (16*(2*tg + s)) times the column rotation (col), and
  // the rotation by one step (kStepTokens) for the query's base position.
  {
    // every table entry of this thread has frequency index j = tid % HALF
    // (kThreads is a multiple of HALF), so one fp64 exp2 serves them all
    static_assert(kThreads % HALF == 0, "table items of a thread share j");
    const int j = tid % HALF;
    const double om = exp2(-(2.0 * j / D) * p.log2_theta);
    const float omf = (float)om;
    if (tid < HALF) {
      float ss, cs;
      sincosf((float)(kStepTokens * om), &ss, &cs);
      rot_s[j] = make_float2(cs, ss);
    }
    for (int i = tid; i < 16 * HALF; i += kThreads) {
      const int c = i / HALF;
      float ss, cs;
      sincosf((float)c * omf, &ss, &cs);
      rope_col[c * 65 + j] = make_float2(cs, ss);
    }
    for (int i = tid; i < 8 * HALF; i += kThreads) {
      const int k = i / HALF;
      float ss, cs;
      sincosf((float)(16.0 * k * om), &ss, &cs);
      rope_ws[k * 64 + j] = make_float2(cs, ss);
    }
  }
  frag_store(w, ld0, live0);
  frag_load(w + kBatch * kWaves, ld1, live1);
  __syncthreads();   // query map, tables
  store_rotated_q<D, NQV>(qc, nql, tid, qo, bs);
  // the lane's fixed key rotations, packed fp16
  CS4 cs[2][NKBS];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int kq = 0; kq < NKBS; ++kq) {
      float cc[4], ss[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = 16 * kq + 4 * quad + e;
        const float2 r = cmul(rope_ws[(2 * tg + s) * 64 + j], rope_col[tcol * 65 + j]);
        cc[e] = r.x;
        ss[e] = r.y;
      }
      cs[s][kq].c01 = __builtin_convertvector((f2){cc[0], cc[1]}, h2);
      cs[s][kq].c23 = __builtin_convertvector((f2){cc[2], cc[3]}, h2);
      cs[s][kq].s01 = __builtin_convertvector((f2){ss[0], ss[1]}, h2);
      cs[s][kq].s23 = __builtin_convertvector((f2){ss[2], ss[3]}, h2);
    }
  frag_store(w + kBatch * kWaves, ld1, live1);
  __syncthreads();   // RoPE tables are dead from here on (the value staging reuses them)
  for (int f0 = w + 2 * kBatch * kWaves; f0 < n_fr; f0 += kBatch * kWaves) {
    u4 ld[kBatch];
    uint32_t live[kBatch];
    frag_load(f0, ld, live);
    frag_store(f0, ld, live);
  }

  // value codes and meta of one step are copied into LDS ahead of use; per-lane
  // offsets of this wave's channel tiles inside a 32-token block
  const int NT = p.rv / 16;
  int v_off[NTW], v_gi[NTW];
  bool v_is8[NTW];
#pragma unroll
  for (int t = 0; t < NTW; ++t) {
    // a wave's tiles beyond the value rank read tile NT-1 (their results are
    // not stored), so the step loop needs no per-tile branch
    const int nt = min(w * NTW + t, NT - 1);
    const int rho = 16 * nt + col;
    const bool is8 = rho < p.v_ro;   // outlier region (8-bit, or 4-bit for MIX4_3)
    if (QM == STARKV_Q_F16) v_off[t] = (rho * 4 + quad) * 16;
    else if (QM == STARKV_Q_MIX4_3)
      v_off[t] = is8 ? (rho * 4 + quad) * 4 : 16 * p.v_ro + ((rho - p.v_ro) * 4 + quad) * 3;
    else if (is8) v_off[t] = (rho * 4 + quad) * 8;
    else v_off[t] = 32 * p.v_ro + ((rho - p.v_ro) * 4 + quad) * 4;
    v_gi[t] = is8 ? rho / 32 : p.v_ng8 + (rho - p.v_ro) / 32;
    v_is8[t] = is8;
  }
  // precision of this wave's value tiles: all 8-bit, all 4-bit (also every
  // INT4 cache), or mixed (only when the 8-bit channel count is not a multiple
  // of 16, or a wave's tiles straddle it); fp16 caches take the first branch
  int vmode = kValues8;
  if (QM != STARKV_Q_F16) {
    bool any8 = false, any4 = false;
    for (int t = 0; t < NTW; ++t) {
      const int nt = min(w * NTW + t, NT - 1);   // the tile the step loop reads
      const bool mix = QM == STARKV_Q_MIX8_4 || QM == STARKV_Q_MIX4_3;
      any8 |= mix && 16 * nt < p.v_ro;
      any4 |= !mix || 16 * nt + 16 > p.v_ro;
    }
    vmode = any8 && any4 ? kValuesMixed : any8 ? kValues8 : kValues4;
  }
  const int vmeta_bytes = 4 * p.v_ng * 128;
  // value copies this wave issues per step (copy_to_lds: one per 8 KB stride)
  auto n_copies = [&](int n_bytes) { return w * 1024 < n_bytes ? (n_bytes - w * 1024 + 8191) / 8192 : 0; };
  const int n_vw = __builtin_amdgcn_readfirstlane(
      n_copies(vcode_bytes) + (QM != STARKV_Q_F16 ? n_copies(vmeta_bytes) : 0));
  auto load_v = [&](int step) {
    const int64_t vblk = step_row(step) >> 5;
    copy_to_lds(vcode, p.cache + p.v_code_off + vblk * 32 * p.v_row_bytes, vcode_bytes, w, lane);
    if (QM != STARKV_Q_F16)
      copy_to_lds(vmeta, p.cache + p.v_meta_off + vblk * p.v_ng * 128, vmeta_bytes, w, lane);
  };
  const uint32_t nib_mask = opaque_u32(0x000F000Fu);

  // ---------------------------------------------------------------- main loop
  float m_run[CTH], l_part[CTH];
  // The two largest scores this lane has seen per tile and subtile (its slot:
  // the tokens 32*tg + 16*s + quad + 4*e of every step), each carrying its
  // token as 4*step + e in the low 8 bits: the combine pass rescores the
  // dominant tokens exactly.
  float b1[CTH][2], b2[CTH][2];
  f4 acc_v[CT][NTW];
#pragma unroll
  for (int c = 0; c < CTH; ++c) {
    m_run[c] = -INFINITY;
    l_part[c] = 0.0f;
    b1[c][0] = b1[c][1] = -INFINITY;
    b2[c][0] = b2[c][1] = -INFINITY;
  }
#pragma unroll
  for (int c = 0; c < CT; ++c)
#pragma unroll
    for (int t = 0; t < NTW; ++t) acc_v[c][t] = (f4){0, 0, 0, 0};

  load_v(0);
  __syncthreads();   // rotated queries of step 0 and the fragments visible

  for (int step = 0; step < n_steps; ++step) {
    const int t_step = t_begin + step * kStepTokens;
    const int tw = t_step + 32 * tg;
    const bool full = (t_step + kStepTokens <= t_end);
    const int64_t kblk_next = (step_row(step + 1) + 32 * tg) >> 4;   // used while step + 1 < n_steps
    // this step's keys were copied before the value copies of the step, which
    // may still be in flight
    wait_vm(n_vw);

    // ------------------------------------------ keys: reconstruct, rotate, score
    f4 acc_s[2][CTH];
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int c = 0; c < CTH; ++c) acc_s[s][c] = (f4){0, 0, 0, 0};
    // nothing pending before the first head: a zero k-block adds nothing
    KeyPending<CTH> pend;
#pragma unroll
    for (int s = 0; s < 2; ++s) { pend.lo[s] = (f4){0, 0, 0, 0}; pend.hi[s] = (f4){0, 0, 0, 0}; }
    pend.q = (h8){0, 0, 0, 0, 0, 0, 0, 0};
    pend.ct = 0;

    // The two waves sharing a SIMD (w and w + 4, one per head half) would
    // split its issue slots unevenly: at equal priority the older wave wins,
    // finishes its heads first and leaves the younger to run its last heads
    // alone, with no second wave to cover its latencies.  With up to two
    // value tiles per wave they take the higher issue priority on alternate
    // heads instead, so that both halves advance together.
#pragma unroll
    for (int k = 1; k <= NKBS; ++k) {
      for (int i = cls_end[k - 1]; i < cls_end[k]; ++i) {
        if constexpr (kAltPrio) {
          if (((i + hh) & 1) != 0) __builtin_amdgcn_s_setprio(1);
          else __builtin_amdgcn_s_setprio(0);
        }
        const HeadRt kh = head_rt(i);
        if constexpr (kPipeKeys) {
          if (k == 1) key_head_q<D, QM, CTH, 1>(kh, raw, frag, qc, qzero, kh.gl, ct0, G, lane, col, tcol, quad, lc4, lc8, cs, acc_s, pend);
          if (k == 2) key_head_q<D, QM, CTH, 2>(kh, raw, frag, qc, qzero, kh.gl, ct0, G, lane, col, tcol, quad, lc4, lc8, cs, acc_s, pend);
          if (NKBS > 2 && k == 3) key_head_q<D, QM, CTH, (NKBS > 2 ? 3 : 1)>(kh, raw, frag, qc, qzero, kh.gl, ct0, G, lane, col, tcol, quad, lc4, lc8, cs, acc_s, pend);
          if (NKBS > 3 && k == 4) key_head_q<D, QM, CTH, (NKBS > 3 ? 4 : 1)>(kh, raw, frag, qc, qzero, kh.gl, ct0, G, lane, col, tcol, quad, lc4, lc8, cs, acc_s, pend);
        } else {
          if (k == 1) key_head<D, QM, CTH, 1>(kh, raw, frag, qc, qzero, kh.gl, ct0, G, lane, col, tcol, quad, cs, acc_s);
          if (k == 2) key_head<D, QM, CTH, 2>(kh, raw, frag, qc, qzero, kh.gl, ct0, G, lane, col, tcol, quad, cs, acc_s);
          if (NKBS > 2 && k == 3) key_head<D, QM, CTH, (NKBS > 2 ? 3 : 1)>(kh, raw, frag, qc, qzero, kh.gl, ct0, G, lane, col, tcol, quad, cs, acc_s);
          if (NKBS > 3 && k == 4) key_head<D, QM, CTH, (NKBS > 3 ? 4 : 1)>(kh, raw, frag, qc, qzero, kh.gl, ct0, G, lane, col, tcol, quad, cs, acc_s);
        }
        // the head's staging has been read (its values are consumed): copy
        // the next step's codes and meta of this head into it
        if (step + 1 < n_steps) copy_head(kh, kblk_next);
      }
    }
    if constexpr (kPipeKeys) key_drain<D, CTH>(pend, cs, acc_s);
    if constexpr (kAltPrio) __builtin_amdgcn_s_setprio(0);
    if constexpr (CTH == 1) {
      // Each half's partial tile holds its own heads' columns and exact zeros
      // in the others (their query operand is zero), so the sum is the tile a
      // single wave would have accumulated over all the heads.
      if (merge) {
        f4* xs = reinterpret_cast<f4*>(smem + LL.xch) + (tg * 64 + lane) * 2;
        if (hh) {
          xs[0] = acc_s[0][0];
          xs[1] = acc_s[1][0];
        }
        lds_barrier();
        if (!hh) {
          acc_s[0][0] += xs[0];
          acc_s[1][0] += xs[1];
        }
      }
    }

    // ------------------------------------------ online softmax (log2 domain)
    // scores are already in log2 units (the query carries log2(e)/sqrt(d))
    // the token of a score (4*step + e, below 256: a split has at most 64
    // steps) replaces the low 8 of its 24 significand bits, a change far below
    // the score's fp16 error; the softmax and the rescoring both use the result
    float x[CTH][2][4];
#pragma unroll
    for (int c = 0; c < CTH; ++c)
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          x[c][s][e] = __uint_as_float((__float_as_uint(acc_s[s][c][e]) & 0xFFFFFF00u) |
                                       (uint32_t)(4 * step + e));
    if (!full) {
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool out = tw + 16 * s + 4 * e + quad >= t_end;
#pragma unroll
          for (int c = 0; c < CTH; ++c) x[c][s][e] = out ? -INFINITY : x[c][s][e];
        }
    }
    // Probabilities are taken against a reference maximum m_run per query
    // column that all waves share without exchanging maxima each step; it is
    // raised (with a rescale of the accumulators) only when a score exceeds it
    // by more than kLazyMargin, so p stays below 2^kLazyMargin.  The first step
    // always sets it.
    bool over = false;
    float ls[CTH];
#pragma unroll
    for (int c = 0; c < CTH; ++c) {
      ls[c] = 0.0f;
      if (c >= ctn) break;
      const int ct = ct0 + c;
      float mx = -INFINITY;
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v = x[c][s][e];
          mx = fmaxf(mx, v);
          b2[c][s] = fmaxf(b2[c][s], fminf(b1[c][s], v));   // the slot's top two
          b1[c][s] = fmaxf(b1[c][s], v);
        }
      mx = wave_max16(mx);
      if (quad == 0) red[(ct * 16 + col) * kTokenGroups + tg] = mx;
      over |= mx > m_run[c] + kLazyMargin;
      const float mr = m_run[c];
      u4 pk;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float e0 = __builtin_amdgcn_exp2f(x[c][k / 2][2 * (k % 2)] - mr);
        const float e1 = __builtin_amdgcn_exp2f(x[c][k / 2][2 * (k % 2) + 1] - mr);
        ls[c] += e0 + e1;
        pk[k] = as_u32(__builtin_convertvector((f2){e0, e1}, h2));
      }
      pbuf[(tg * CT + ct) * 64 + lane] = __builtin_bit_cast(h8, pk);
    }
    const bool any_over = __any(over);
    if (lane == 0) flag_s[w] = any_over ? 1 : 0;
    // this wave's value copies landed (the next step's key copies, issued after
    // them, may still be in flight)
    wait_vm(step + 1 < n_steps ? n_kw : 0);
    lds_barrier();   // (1) probabilities, maxima, flags and the step's values visible
    if (step + 1 < n_steps) {   // every wave is done with the queries: rotate them
      const int j0 = 4 * (tid % (D / 8));
#pragma unroll
      for (int e = 0; e < 4; ++e) bs[e] = cmul(bs[e], rot_s[j0 + e]);
      store_rotated_q<D, NQV>(qc, nql, tid, qo, bs);
    }
    const int4 f0 = *reinterpret_cast<const int4*>(flag_s);
    const int4 f1 = *reinterpret_cast<const int4*>(flag_s + 4);
    if ((f0.x | f0.y | f0.z | f0.w | f1.x | f1.y | f1.z | f1.w) != 0) {
      // raise the reference of every column to the running maximum and redo
      // this step's probabilities against it
#pragma unroll
      for (int c = 0; c < CTH; ++c) {
        if (c >= ctn) break;
        const int ct = ct0 + c;
        const f4 tm = *reinterpret_cast<const f4*>(red + (ct * 16 + col) * kTokenGroups);
        const float mn = fmaxf(fmaxf(m_run[c], fmaxf(tm[0], tm[1])), fmaxf(tm[2], tm[3]));
        const float al = __builtin_amdgcn_exp2f(m_run[c] - mn);   // m_run = -inf first: 0
        m_run[c] = mn;
        u4 pk;
        float l2 = 0.0f;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float e0 = __builtin_amdgcn_exp2f(x[c][k / 2][2 * (k % 2)] - mn);
          const float e1 = __builtin_amdgcn_exp2f(x[c][k / 2][2 * (k % 2) + 1] - mn);
          l2 += e0 + e1;
          pk[k] = as_u32(__builtin_convertvector((f2){e0, e1}, h2));
        }
        l_part[c] = l_part[c] * al + l2;
        pbuf[(tg * CT + ct) * 64 + lane] = __builtin_bit_cast(h8, pk);
        if (tg == 0 && quad == 0) alpha_s[ct * 16 + col] = al;
      }
      lds_barrier();   // new probabilities and rescale factors visible
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const f4 al = *reinterpret_cast<const f4*>(alpha_s + c * 16 + 4 * quad);
#pragma unroll
        for (int t = 0; t < NTW; ++t) acc_v[c][t] *= al;
      }
    } else {
#pragma unroll
      for (int c = 0; c < CTH; ++c) l_part[c] += ls[c];
    }

    // ------------------------------------------ values: acc += P . V'
    // The precision of a wave's value tiles does not change between steps, so
    // the wave runs one branch-free variant (see vmode) and the loads of all
    // token groups can be issued ahead of the dequantization.
    auto values = [&](auto vm_tag, auto full_tag) {
      constexpr int VM = decltype(vm_tag)::value;
      constexpr bool FULL = decltype(full_tag)::value;
#pragma unroll
      for (int ww = 0; ww < kTokenGroups; ++ww) {
        h8 pa[CT];
#pragma unroll
        for (int c = 0; c < CT; ++c) pa[c] = pbuf[(ww * CT + c) * 64 + lane];
        // slots 2k, 2k+1 of this lane's chunk: tokens
        //   k < 2: quad + 8k + {0,4};  k >= 2: 16 + quad + 8(k-2) + {0,4}
        u4 vmask;
        if (!FULL) {
          const int tb = t_step + 32 * ww;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int t0 = tb + quad + (k < 2 ? 8 * k : 16 + 8 * (k - 2));
            vmask[k] = (t0 < t_end ? 0x0000FFFFu : 0u) | (t0 + 4 < t_end ? 0xFFFF0000u : 0u);
          }
        }
        const uint8_t* vb = vcode + ww * 32 * p.v_row_bytes;
#pragma unroll
        for (int t = 0; t < NTW; ++t) {
          u4 v;
          if (QM == STARKV_Q_F16) {
            v = *reinterpret_cast<const u4*>(vb + v_off[t]);
          } else {
            const uint8_t* mb = vmeta + ((ww * p.v_ng + v_gi[t]) * 4 + quad) * 32;
            const u4 sv = *reinterpret_cast<const u4*>(mb);
            const u4 zv = *reinterpret_cast<const u4*>(mb + 16);
            if (QM == STARKV_Q_MIX4_3) {
              // outlier tiles: one 4-bit word per lane; inlier tiles: 3 bytes
              // (slot pairs 2k, 2k+1 at fields k, k+4 of the 24-bit word)
              const uint32_t d = VM == kValues8 ? *reinterpret_cast<const uint32_t*>(vb + v_off[t])
                                                : lds_word_at(vb, v_off[t]);
              const u4 v4 = deq_int4m(d, nib_mask, as_h2(sv.x), as_h2(zv.x), as_h2(sv.y),
                                      as_h2(zv.y), as_h2(sv.z), as_h2(zv.z), as_h2(sv.w),
                                      as_h2(zv.w));
              const u4 m3 = magic_int3(d);
              const u4 v3 = (u4){deq_pair(m3.x, as_h2(sv.x), as_h2(zv.x)),
                                 deq_pair(m3.y, as_h2(sv.y), as_h2(zv.y)),
                                 deq_pair(m3.z, as_h2(sv.z), as_h2(zv.z)),
                                 deq_pair(m3.w, as_h2(sv.w), as_h2(zv.w))};
              v = VM == kValues8 ? v4 : VM == kValues4 ? v3 : (v_is8[t] ? v4 : v3);
            } else if (VM == kValues8) {
              const u2 d = *reinterpret_cast<const u2*>(vb + v_off[t]);
              v = deq_int8p(d, as_h2(sv.x), as_h2(zv.x), as_h2(sv.y), as_h2(zv.y), as_h2(sv.z),
                            as_h2(zv.z), as_h2(sv.w), as_h2(zv.w));
            } else if (VM == kValues4) {
              const uint32_t d = *reinterpret_cast<const uint32_t*>(vb + v_off[t]);
              v = deq_int4m(d, nib_mask, as_h2(sv.x), as_h2(zv.x), as_h2(sv.y), as_h2(zv.y),
                            as_h2(sv.z), as_h2(zv.z), as_h2(sv.w), as_h2(zv.w));
            } else {
              // 8-bit and 4-bit lanes in one wave: an aligned 8-byte read
              // serves both (a 4-bit lane takes the half holding its word)
              const u2 d = *reinterpret_cast<const u2*>(vb + (v_off[t] & ~7));
              const uint32_t d4 = (v_off[t] & 4) ? d.y : d.x;
              const u4 v8 = deq_int8p(d, as_h2(sv.x), as_h2(zv.x), as_h2(sv.y), as_h2(zv.y),
                                      as_h2(sv.z), as_h2(zv.z), as_h2(sv.w), as_h2(zv.w));
              const u4 v4 = deq_int4m(d4, nib_mask, as_h2(sv.x), as_h2(zv.x), as_h2(sv.y),
                                      as_h2(zv.y), as_h2(sv.z), as_h2(zv.z), as_h2(sv.w),
                                      as_h2(zv.w));
              v = v_is8[t] ? v8 : v4;
            }
          }
          if (!FULL) v &= vmask;
          const h8 vop = __builtin_bit_cast(h8, v);
#pragma unroll
          for (int c = 0; c < CT; ++c) acc_v[c][t] = mfma16(pa[c], vop, acc_v[c][t]);
        }
      }
    };
    using Full = std::true_type;
    if (!full) values(std::integral_constant<int, kValuesMixed>{}, std::false_type{});
    else if (vmode == kValues8) values(std::integral_constant<int, kValues8>{}, Full{});
    else if (vmode == kValues4) values(std::integral_constant<int, kValues4>{}, Full{});
    else values(std::integral_constant<int, kValuesMixed>{}, Full{});
    if (step + 1 < n_steps) {
      lds_barrier();   // every wave is done reading this step's values
      load_v(step + 1);
    }
  }

  // ---------------------------------------------------------------- partials
#pragma unroll
  for (int c = 0; c < CTH; ++c) {
    if (c >= ctn) break;
    const float l = wave_sum16(l_part[c]);
    if (quad == 0) red[((ct0 + c) * 16 + col) * kTokenGroups + tg] = l;
  }
  __syncthreads();
  const int64_t pbase = (int64_t)pitem * p.n_q;
  // Candidates of a query head, in blocks of the 16 entries of one wave.  With
  // m and l this split's maximum and normalizer and M, L the merged ones, a
  // score x has the rescoring priority 2^(x - M) (1 + |x|) / L, at most
  // 2^(m - M) q / L with q = max over the block of 2^(x - m) (1 + |x|), and at
  // most q / l (L >= 2^(m - M) l).  So a block whose q misses half the
  // threshold times l is never rescored and is not written; partial slot
  // rv + 2 holds a byte per block saying whether it was, rv + 4 + tg the
  // block's q, from which the merge bounds the block before loading it.
#pragma unroll
  for (int c = 0; c < CTH; ++c) {
    if (c >= ctn) break;
    const int il = (ct0 + c) * 16 + col;
    const f4 lg = *reinterpret_cast<const f4*>(red + il * kTokenGroups);
    const float bar = 0.5f * kRescoreTau * (((lg[0] + lg[1]) + lg[2]) + lg[3]);
    const float mr = m_run[c];
    auto bound = [&](float v) {
      return v == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(v - mr) * (1.0f + fabsf(v));
    };
    float qb = fmaxf(fmaxf(bound(b1[c][0]), bound(b2[c][0])), fmaxf(bound(b1[c][1]), bound(b2[c][1])));
    qb = fmaxf(qb, __shfl_xor(qb, 16));
    qb = fmaxf(qb, __shfl_xor(qb, 32));
    const bool any = qb >= bar;
    if (il < nql && quad == 0) {
      float* slot = p.part + (pbase + qmap[il]) * p.part_stride + p.rv;
      reinterpret_cast<uint8_t*>(slot + 2)[tg] = any ? 1 : 0;
      slot[4 + tg] = qb;
    }
    if (il < nql && any) {
      float2* cd = p.cand + (pbase + qmap[il]) * kCand + (tg * 4 + quad) * 4;
      auto token = [&](float v, int s) {
        const uint32_t k = __float_as_uint(v) & 0xFFu;
        return __int_as_float(t_begin + (int)(k >> 2) * kStepTokens + 4 * (int)(k & 3u) + 16 * s +
                              32 * tg + quad);
      };
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        cd[2 * s] = make_float2(b1[c][s], token(b1[c][s], s));
        cd[2 * s + 1] = make_float2(b2[c][s], token(b2[c][s], s));
      }
    }
  }
  if (tg == 0 && quad == 0) {
#pragma unroll
    for (int c = 0; c < CTH; ++c) {
      if (c >= ctn) break;
      const int il = (ct0 + c) * 16 + col;
      if (il < nql) {
        float lt = 0.0f;
#pragma unroll
        for (int g = 0; g < kTokenGroups; ++g) lt += red[((ct0 + c) * 16 + col) * kTokenGroups + g];
        float* dst = p.part + (pbase + qmap[il]) * p.part_stride + p.rv;
        dst[0] = m_run[c];
        dst[1] = lt;
      }
    }
  }
#pragma unroll
  for (int c = 0; c < CT; ++c)
#pragma unroll
    for (int t = 0; t < NTW; ++t) {
      const int nt = w * NTW + t;
      if (nt < NT) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int il = c * 16 + 4 * quad + e;
          if (il < nql) p.part[(pbase + qmap[il]) * p.part_stride + 16 * nt + col] = acc_v[c][t][e];
        }
      }
    }
}

// ---------------------------------------------------------------------- combine
#ifdef SK_COMMON
// One workgroup per (query head, sequence), or two that each up-project half
// of the output columns when the grid is small.  Merges the splits with weights
// 2^(m_s - M), corrects the few tokens that dominate the softmax with exactly
// recomputed scores, and applies the value up-projection of the head's KV group.
// All loads of a phase are issued before their results are used, so each phase
// costs about one memory round trip.
//
// Exact rescoring.  The split pass scores with fp16 rotated keys and fp16
// dequantized latents; the relative error of a score is a few fp16 ulps, so a
// token's weight is off by about (score magnitude) x 2^-11.  That only matters
// for tokens holding a large share of the softmax mass, and the split pass
// reports the two largest approximate scores of every lane (kCand per split and
// query head).  Candidates whose share times (1 + |score|) reaches kRescoreTau
// are recomputed here in fp32 from the cache (fp32 dequantization, fp32
// reconstruction, RoPE angle reduced in fp64), and their contribution to the
// normalizer and to the merged value latent is moved from the approximate to the
// exact weight.
constexpr int kCombineMaxSplits = 256;  // one split per thread of the weight pass
constexpr int kRescoreMax = 128;                       // tokens rescored per query head
constexpr int kRescoreBatch = 32;                      // of them with key latents in LDS at once
constexpr int kBkVecPerThread = 8;   // B_k block of up to 128 x 128 fp16: 2048 vectors / 256 threads
// candidate entries are read in chunks of 64 splits, kCandPerThread per thread
constexpr int kCandChunk = 64 * kCand;
constexpr int kCandPerThread = kCandChunk / 256;

__device__ __forceinline__ float h2f(uint16_t u) { return (float)__builtin_bit_cast(_Float16, u); }

// Dequantized key latent channel ch of head g at token t of sequence b.
// bits of the outlier and inlier regions of a quantized cache
__device__ __forceinline__ int region_hi_bits(int qmode) { return qmode == STARKV_Q_MIX8_4 ? 8 : 4; }
__device__ __forceinline__ int region_lo_bits(int qmode) { return qmode == STARKV_Q_MIX4_3 ? 3 : 4; }

// `bits`-wide field at bit `sh` of the little-endian word starting at w (the
// word's bytes are read one at a time: 3-bit words are not aligned)
__device__ __forceinline__ int code_field(const uint8_t* w, int sh, int bits) {
  const int b0 = sh / 8;
  uint32_t v = w[b0];
  if (sh % 8 + bits > 8) v |= (uint32_t)w[b0 + 1] << 8;
  return (int)((v >> (sh % 8)) & ((1u << bits) - 1));
}

__device__ float key_latent(const CombineParams& p, int g, int b, int t, int ch) {
  const int64_t blk = cache_row(p.rmap, b, t) / 16;
  const int tau = t % 16, c = ch / 8, wi = ch % 8;
  const uint8_t* code = p.cache + p.k_code_off[g] + blk * 16 * p.k_rb[g];
  if (p.qmode == STARKV_Q_F16)
    return h2f(*reinterpret_cast<const uint16_t*>(code + c * 256 + tau * 16 + wi * 2));
  const int ro = p.k_ro[g], nhi = ro / 8;
  const int hb = region_hi_bits(p.qmode), lb = region_lo_bits(p.qmode);
  const bool hi = ch < ro;
  const int bits = hi ? hb : lb;
  // chunk c: 16 tokens x `bits` bytes, outlier chunks first; channel wi at bits*wi
  const uint8_t* tok = code + (hi ? c * 16 * hb : nhi * 16 * hb + (c - nhi) * 16 * lb) + tau * bits;
  const int q = bits == 8 ? tok[wi] : code_field(tok, bits * wi, bits);
  const int grp = hi ? ch / 32 : (ro + 31) / 32 + (ch - ro) / 32;
  const uint16_t* m = reinterpret_cast<const uint16_t*>(
      p.cache + p.k_meta_off[g] + (blk * p.k_ng[g] + grp) * 64 + tau * 4);
  return __builtin_fmaf((float)q, h2f(m[0]), h2f(m[1]));
}

// Dequantized value latent channel r at token t of sequence b.
__device__ float value_latent(const CombineParams& p, int b, int t, int r) {
  const int64_t blk = cache_row(p.rmap, b, t) / 32;
  const int u = t % 32, kq = u % 4, slot = 4 * (u / 16) + (u % 16) / 4;
  const uint8_t* code = p.cache + p.v_code_off + blk * 32 * p.v_rb;
  if (p.qmode == STARKV_Q_F16)
    return h2f(*reinterpret_cast<const uint16_t*>(code + (r * 4 + kq) * 16 + slot * 2));
  const int hb = region_hi_bits(p.qmode), lb = region_lo_bits(p.qmode);
  const bool hi = r < p.v_ro;
  const int bits = hi ? hb : lb;
  // (channel, chunk) words of `bits` bytes, the outlier region first
  const uint8_t* wd = code + (hi ? (r * 4 + kq) * hb : 4 * p.v_ro * hb + ((r - p.v_ro) * 4 + kq) * lb);
  int q;
  if (bits == 8) {
    q = wd[slot];
  } else {
    // slot 2k / 2k+1 at fields k / k+4 of the word (4 bits: 4 bits apiece and the
    // second half at bit 16; 3 bits: 3 bits apiece and the second half at bit 12)
    const int sh = bits == 4 ? ((slot & 1) ? 16 + 4 * (slot / 2) : 4 * (slot / 2))
                             : ((slot & 1) ? 12 + 3 * (slot / 2) : 3 * (slot / 2));
    q = code_field(wd, sh, bits);
  }
  const int grp = hi ? r / 32 : (p.v_ro + 31) / 32 + (r - p.v_ro) / 32;
  const uint8_t* m = p.cache + p.v_meta_off + blk * p.v_ng * 128 + (grp * 4 + kq) * 32;
  return __builtin_fmaf((float)q, h2f(reinterpret_cast<const uint16_t*>(m)[slot]),
                        h2f(reinterpret_cast<const uint16_t*>(m + 16)[slot]));
}

// floats of the combine kernel's LDS before its shared region (kept a multiple
// of 4 so that the region is 16-byte aligned)
__host__ __device__ constexpr int combine_head_floats(int rv) {
  return (rv + 2 * kCombineMaxSplits + 3 * kRescoreMax + 16 + 3) / 4 * 4;
}

// DEEP (grids of at most one workgroup per compute unit): both partial batches
// of the first 64 splits and the thread's U_V rows are loaded at entry.
// Otherwise (several workgroups per compute unit) the second batch is loaded
// when needed and U_V just before the merge, which keeps the kernel at 128
// VGPRs (four workgroups per compute unit).
template <bool DEEP>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(DEEP ? 1 : 4)))
void decode_combine_kernel(CombineParams p) {
  extern __shared__ __align__(16) float sm[];
  const int D = p.head_dim;
  float* a = sm;                         // [rv] merged value latent
  float* wts = a + p.rv;                 // [kCombineMaxSplits] split weights
  float* c_x = wts + kCombineMaxSplits;  // [kRescoreMax] approximate scores
  float* c_d = c_x + kRescoreMax;        // [kRescoreMax] weight corrections
  int* c_t = reinterpret_cast<int*>(c_d + kRescoreMax);   // [kRescoreMax] tokens
  uint32_t* sfl = reinterpret_cast<uint32_t*>(c_t + kRescoreMax);  // [kCombineMaxSplits] flags
  float* misc = reinterpret_cast<float*>(sfl + kCombineMaxSplits);  // M, L, L', unused
  float* wmax = misc + 4;                // [4] per-wave split maxima
  float* wsum = misc + 8;                // [4] per-wave weighted sums
  int* wfl = reinterpret_cast<int*>(misc + 12);   // [4] per-wave: a split flagged candidates
  // One region, 16-byte aligned, serves two phases: the merge (per-wave split
  // sums, and the rescoring's key latents and B_k block) and, once the merged
  // latent is in `a`, the up-projection's partial sums.
  float* uni = sm + combine_head_floats(p.rv);
  float* red4 = uni;                                   // [4][rv] per-wave split sums
  float* lat = red4 + 4 * p.rv;                        // [kRescoreBatch][rmax] key latents
  uint16_t* bks = reinterpret_cast<uint16_t*>(lat + kRescoreBatch * p.rmax);  // [rmax][D] fp16
  float* red = uni;                                    // [256 / (D/8)][D] partial up-projections
  const int i = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  // output columns c_0 .. c_0 + Dc - 1 of this workgroup (the merge and the
  // rescoring are repeated by each of the col_split workgroups of the head)
  const int Dc = D / p.col_split, c_0 = blockIdx.z * Dc;
  const int lane = tid & 63, w = tid >> 6;
  const int g = (int)(((int64_t)i * p.n_kv) / p.n_q);
  // this sequence's splits: under the work plan, items first .. first + ns - 1
  // (the split pass wrote the plan), else the fixed split grid
  int L, ns, first;
  if (p.dyn) {
    const int4 e = *reinterpret_cast<const int4*>(p.plan + 4 * b);
    first = e.x;
    ns = e.y;
    L = e.z;
  } else {
    L = p.ctx_len[b];
    L = L < 0 ? 0 : (L > p.max_ctx ? p.max_ctx : L);
    ns = (L + p.split_len - 1) / p.split_len;
    first = b * p.n_split;
  }
  const int64_t out_row = ((int64_t)b * p.n_q + i) * D;
  const bool to_lat = p.lat != nullptr;
  const int64_t lat_row = ((int64_t)b * p.n_q + i) * p.rv;
  const int64_t lat_lo = (int64_t)p.batch * p.n_q * p.rv;
  if (L == 0) {
    if (to_lat) {
      for (int r = tid; r < p.rv; r += 256) p.lat[lat_row + r] = p.lat[lat_lo + lat_row + r] = 0;
      return;
    }
    for (int j = c_0 + tid; j < c_0 + Dc; j += 256) {
      if (p.out_dtype == STARKV_DT_F32) static_cast<float*>(p.out)[out_row + j] = 0.0f;
      else static_cast<uint16_t*>(p.out)[out_row + j] = 0;
    }
    return;
  }
  const float* part = p.part + ((int64_t)first * p.n_q + i) * p.part_stride;
  const int64_t sstride = (int64_t)p.n_q * p.part_stride;
  // Every load that does not depend on the split weights is issued at once so
  // that they share one memory round trip: each split's maximum, normalizer and
  // candidate flags (one split per thread), the value-latent partials of the
  // first 64 splits and this thread's first rows of U_V.
  // (m, l, flags, unused) and the four block bounds: two 16-byte loads from a
  // valid split, not in a branch, so that the first wait covers only them
  const float* ps = part + min(tid, ns - 1) * sstride + p.rv;
  const f4 ml0 = *reinterpret_cast<const f4*>(ps);
  const f4 qb0 = *reinterpret_cast<const f4*>(ps + 4);
  const float mv0 = tid < ns ? ml0[0] : -INFINITY;
  const float lv0 = ml0[1];
  const uint32_t fl0 = tid < ns ? __float_as_uint(ml0[2]) : 0u;
  const int D8 = Dc / 8;                 // 16, 8 or 4 column vectors
  const int groups = 256 / D8;           // row groups of the up-projection
  const int j8 = tid % D8, rg = tid / D8;
  const int64_t ldb = (int64_t)p.n_kv * D;
  const uint16_t* bv = p.bv + (int64_t)g * D + c_0 + 8 * j8;
  // 32-bit byte offsets from the (b, head) partials: the region spans
  // n_split * sstride floats, far below 4 GiB
  const uint8_t* pbase = reinterpret_cast<const uint8_t*>(part);
  const uint32_t sbytes = (uint32_t)sstride * 4u;
  // Value-latent partials: wave w takes splits w, w + 4, .., lane l channels
  // 4l..4l+3 of each 256-channel chunk, one 16-byte load per (split, chunk), so
  // a chunk of all splits is 64 loads of 1 KiB per workgroup.  A wave loads its
  // splits in batches of 8 (splits w + 32h + 4k); the two batches of chunk 0
  // (splits below 64) are loaded now.
  constexpr int kSplitBatch = 8;
  const int n_chunk = (p.rv + 255) / 256;
  auto load_batch = [&](int ch, int h, f4 (&pv)[kSplitBatch]) {
    const uint32_t o = (uint32_t)min(256 * ch + 4 * lane, p.rv - 4) * 4u;
#pragma unroll
    for (int k = 0; k < kSplitBatch; ++k)
      pv[k] = *reinterpret_cast<const f4*>(
          pbase + o + (uint32_t)min(w + 32 * h + 4 * k, ns - 1) * sbytes);
  };
  f4 pv0[kSplitBatch], pv1[kSplitBatch];
  load_batch(0, 0, pv0);
  if constexpr (DEEP) load_batch(0, 1, pv1);   // (clamped split indices: valid, unused below 33 splits)
  // rows of U_V per thread per round of loads: 8 when they are loaded at entry,
  // 16 when loaded before the merge (then the partials' registers are free)
  constexpr int kUpRows = DEEP ? 8 : 16;
  // rows past rv load row rv - 1 and are skipped by the product.  The loads are
  // not in a branch, so that no wait before them covers more than it must: with
  // latent output (no U_V) they read the first partials, unused.
  const uint16_t* bvl = to_lat ? reinterpret_cast<const uint16_t*>(part) : bv;
  const int64_t ldbl = to_lat ? 0 : ldb;
  auto load_rows = [&](int r0, u4 (&w8)[kUpRows]) {
#pragma unroll
    for (int k = 0; k < kUpRows; ++k)
      w8[k] = *reinterpret_cast<const u4*>(bvl + (int64_t)min(r0 + k * groups, p.rv - 1) * ldbl);
  };
  u4 w0[kUpRows];
  if constexpr (DEEP) load_rows(rg, w0);
  const int r_g = p.k_rank[g];
  {                               // split weights: one split per thread
    float m = mv0;
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    if (lane == 0) wmax[w] = m;
    __syncthreads();
    m = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
    const float wv = tid < ns ? __builtin_amdgcn_exp2f(mv0 - m) : 0.0f;
    wts[tid] = wv;
    float l = tid < ns ? wv * lv0 : 0.0f;
    for (int o = 32; o > 0; o >>= 1) l += __shfl_xor(l, o);
    if (lane == 0) wsum[w] = l;
    __syncthreads();
    const float ls = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
    // the candidate blocks of this split that may hold a token to rescore:
    // written by the split and bounded by 2^(m_s - M) q / L >= tau / 2
    uint32_t fl = 0;
#pragma unroll
    for (int t = 0; t < 4; ++t)
      if (((fl0 >> (8 * t)) & 0xFFu) != 0u && wv * qb0[t] >= 0.5f * kRescoreTau * ls)
        fl |= 1u << (8 * t);
    sfl[tid] = fl;
    const bool fw = __ballot(fl != 0u) != 0;
    if (lane == 0) wfl[w] = fw ? 1 : 0;
    if (tid == 0) { misc[0] = m; misc[1] = ls; }
    __syncthreads();
  }
  const float M = misc[0], Lsum = misc[1];
  const bool any_cand = (wfl[0] | wfl[1] | wfl[2] | wfl[3]) != 0;
  // weighted sums of this wave's splits, per channel, into red4[w][r]
  auto add_batch = [&](int h, const f4 (&pv)[kSplitBatch], f4& acc) {
#pragma unroll
    for (int k = 0; k < kSplitBatch; ++k) {
      const int sp = w + 32 * h + 4 * k;
      if (sp < ns) acc += wts[sp] * pv[k];
    }
  };
  for (int ch = 0; ch < n_chunk; ++ch) {
    f4 acc = (f4){0, 0, 0, 0};
    if (ch == 0) {
      add_batch(0, pv0, acc);
      if (ns > 32) {                           // splits 32 .. 63
        if constexpr (DEEP) {
          add_batch(1, pv1, acc);
        } else {
          load_batch(0, 1, pv1);
          add_batch(1, pv1, acc);
        }
      }
    } else {
      f4 pa[kSplitBatch], pb[kSplitBatch];
      load_batch(ch, 0, pa);
      if (ns > 32) load_batch(ch, 1, pb);
      add_batch(0, pa, acc);
      if (ns > 32) add_batch(1, pb, acc);
    }
    const int r = 256 * ch + 4 * lane;
    if (r < p.rv) *reinterpret_cast<f4*>(red4 + w * p.rv + r) = acc;
  }
  // splits beyond 64 (long sequences): further batches added to the wave's own
  // partial sums, in the same order
  for (int h = 2; 32 * h < ns; ++h)
    for (int ch = 0; ch < n_chunk; ++ch) {
      f4 pv[kSplitBatch];
      load_batch(ch, h, pv);
      const int r = 256 * ch + 4 * lane;
      if (r < p.rv) {
        f4 acc = *reinterpret_cast<const f4*>(red4 + w * p.rv + r);
        add_batch(h, pv, acc);
        *reinterpret_cast<f4*>(red4 + w * p.rv + r) = acc;
      }
    }

  // ---- candidate selection: share x (1 + |x|) >= tau, tau raised by 4 until
  // at most kRescoreMax remain (at most 8 thresholds); compaction in entry
  // order (deterministic).  Up to 64 splits the entries stay in registers;
  // beyond, one pass over the chunks counts the entries above each threshold
  // and a second compacts, reading the chunks again.
  constexpr int kLevels = 8;
  // Candidate entries of the splits.  Thread tid takes slot `lane` of splits
  // 64 c + 4 k + w of chunk c (entry order: split, then slot); a slot's block of
  // 16 entries holds data only when the split set its flag byte, and the rest
  // read as -inf scores (never selected).
  static_assert(kCand == 64 && kCandPerThread == 16, "one slot per lane");
  const float2* cand = p.cand + ((int64_t)first * p.n_q + i) * kCand;
  auto load_cand = [&](int c, float2 (&ce)[kCandPerThread]) {
    const float2* cl = cand + (int64_t)(64 * c + w) * p.n_q * kCand + lane;
    const int64_t cstep = (int64_t)4 * p.n_q * kCand;
#pragma unroll
    for (int k = 0; k < kCandPerThread; ++k) {
      const int s = 64 * c + 4 * k + w;
      ce[k] = make_float2(-INFINITY, 0.0f);
      if (s < ns && ((sfl[s] >> (8 * (lane >> 4))) & 0xFFu) != 0u) ce[k] = cl[k * cstep];
    }
  };
  const int n_cchunk = (ns + 63) / 64;
  auto priorities = [&](const float2 (&ce)[kCandPerThread], float (&prio)[kCandPerThread]) {
#pragma unroll
    for (int k = 0; k < kCandPerThread; ++k) {
      const float x = ce[k].x;
      prio[k] = (x == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(x - M) / Lsum * (1.0f + fabsf(x));
    }
  };
  int* kcnt = reinterpret_cast<int*>(lat);   // [kCandPerThread][4] wave counts (lat is free here)
  // one chunk's entries with prio >= tau go to c_x / c_t from `base` on, in
  // entry order; returns the next base
  auto compact = [&](const float2 (&ce)[kCandPerThread], const float (&prio)[kCandPerThread],
                     float tau, int base) {
    uint64_t bal[kCandPerThread];
#pragma unroll
    for (int k = 0; k < kCandPerThread; ++k) {
      bal[k] = __ballot(prio[k] >= tau);
      if (lane == 0) kcnt[4 * k + w] = __builtin_popcountll(bal[k]);
    }
    __syncthreads();
    // the wave counts of four entries at a time, read together
#pragma unroll
    for (int k0 = 0; k0 < kCandPerThread; k0 += 4) {
      int4 kc[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) kc[j] = *reinterpret_cast<const int4*>(kcnt + 4 * (k0 + j));
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int k = k0 + j;
        const int off = base + (w > 0 ? kc[j].x : 0) + (w > 1 ? kc[j].y : 0) + (w > 2 ? kc[j].z : 0);
        if (prio[k] >= tau) {
          const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal[k] >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)bal[k], 0));
          if (off + rank < kRescoreMax) {
            c_x[off + rank] = ce[k].x;
            c_t[off + rank] = __float_as_int(ce[k].y);
          }
        }
        base += kc[j].x + kc[j].y + kc[j].z + kc[j].w;
      }
    }
    __syncthreads();                     // kcnt is rewritten by the next chunk
    return base;
  };
  float tau = kRescoreTau;
  int n_sel = 0;
  if (!any_cand) {
    // no split holds a candidate that could reach the threshold
  } else if (n_cchunk == 1) {
    float2 ce0[kCandPerThread];
    load_cand(0, ce0);
    float prio[kCandPerThread];
    priorities(ce0, prio);
    {
      int c = 0;
#pragma unroll
      for (int k = 0; k < kCandPerThread; ++k) c += prio[k] >= tau;
      for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
      if (lane == 0) kcnt[w] = c;
      __syncthreads();
      n_sel = kcnt[0] + kcnt[1] + kcnt[2] + kcnt[3];
      __syncthreads();
    }
    if (n_sel > kRescoreMax) {
      // the higher thresholds counted in one pass (16-bit fields, as for
      // several chunks below), then the first that leaves at most kRescoreMax
      uint32_t lv[kLevels / 2];
#pragma unroll
      for (int j = 0; j < kLevels / 2; ++j) lv[j] = 0;
#pragma unroll
      for (int k = 0; k < kCandPerThread; ++k) {
        float t = kRescoreTau;
#pragma unroll
        for (int j = 0; j < kLevels; ++j, t *= 4.0f)
          lv[j / 2] += prio[k] >= t ? 1u << (16 * (j % 2)) : 0u;
      }
#pragma unroll
      for (int j = 0; j < kLevels / 2; ++j) {
        uint32_t v = lv[j];
        for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
        if (lane == 0) kcnt[4 * j + w] = (int)v;
      }
      __syncthreads();
      for (int j = 1; j < kLevels; ++j) {
        tau *= 4.0f;
        n_sel = 0;
        for (int ww = 0; ww < 4; ++ww) n_sel += ((uint32_t)kcnt[4 * (j / 2) + ww] >> (16 * (j % 2))) & 0xFFFFu;
        if (n_sel <= kRescoreMax) break;
      }
      __syncthreads();                   // the counts are read before kcnt is rewritten
    }
    // past the cap at every threshold tried (at least kRescoreMax tokens each
    // holding that much): the first kRescoreMax of the last one, in entry order
    if (n_sel > 0) compact(ce0, prio, tau, 0);
    n_sel = min(n_sel, kRescoreMax);
  } else {
    // entries at or above threshold j, per thread, in 16-bit fields (field j % 2
    // of word j / 2; at most 32 per thread and 2048 per wave)
    uint32_t lv[kLevels / 2];
#pragma unroll
    for (int j = 0; j < kLevels / 2; ++j) lv[j] = 0;
    for (int c = 0; c < n_cchunk; ++c) {
      float2 ce[kCandPerThread];
      load_cand(c, ce);
      float prio[kCandPerThread];
      priorities(ce, prio);
#pragma unroll
      for (int k = 0; k < kCandPerThread; ++k) {
        float t = kRescoreTau;
#pragma unroll
        for (int j = 0; j < kLevels; ++j, t *= 4.0f)
          lv[j / 2] += prio[k] >= t ? 1u << (16 * (j % 2)) : 0u;
      }
    }
#pragma unroll
    for (int j = 0; j < kLevels / 2; ++j) {
      uint32_t v = lv[j];
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
      if (lane == 0) kcnt[4 * j + w] = (int)v;
    }
    __syncthreads();
    for (int j = 0; j < kLevels; ++j) {
      n_sel = 0;
      for (int ww = 0; ww < 4; ++ww) n_sel += ((uint32_t)kcnt[4 * (j / 2) + ww] >> (16 * (j % 2))) & 0xFFFFu;
      if (n_sel <= kRescoreMax || j == kLevels - 1) break;
      tau *= 4.0f;
    }
    __syncthreads();                     // the counts are read before kcnt is rewritten
    if (n_sel > 0) {
      int base = 0;
      for (int c = 0; c < n_cchunk; ++c) {
        float2 ce[kCandPerThread];
        load_cand(c, ce);
        float prio[kCandPerThread];
        priorities(ce, prio);
        base = compact(ce, prio, tau, base);
      }
    }
    n_sel = min(n_sel, kRescoreMax);
  }
  if (n_sel > 0) {
    // one round of loads for the rescoring: the KV head's up-projection block
    // B_k (r_g x D fp16, staged in LDS) and the candidates' key latents
    const int nbk = r_g * D / 8;           // 16-byte vectors
    u4 bkv[kBkVecPerThread];
    {
      const u4* src = reinterpret_cast<const u4*>(p.bk + (int64_t)p.k_bkrow[g] * D);
#pragma unroll
      for (int k = 0; k < kBkVecPerThread; ++k)
        bkv[k] = src[min(tid + k * 256, nbk - 1)];
    }
#pragma unroll
    for (int k = 0; k < kBkVecPerThread; ++k)
      if (tid + k * 256 < nbk) reinterpret_cast<u4*>(bks)[tid + k * 256] = bkv[k];
    // ---- exact scores, kRescoreBatch candidates at a time: their dequantized
    // key latents, then one (candidate, RoPE pair) item per thread; the items of
    // a candidate are consecutive lanes of one wave and are summed with shuffles
    const int HALF = D / 2;
    const uint16_t* bk = bks;
    const uint16_t* qs = static_cast<const uint16_t*>(p.q) + ((int64_t)b * p.n_q + i) * D;
    for (int j0 = 0; j0 < n_sel; j0 += kRescoreBatch) {
    const int nb = min(kRescoreBatch, n_sel - j0);
    if (j0 > 0) __syncthreads();         // the previous batch's latents are read
    for (int it = tid; it < nb * r_g; it += 256) {
      const int j = it / r_g, ch = it % r_g;
      lat[j * p.rmax + ch] = key_latent(p, g, b, c_t[j0 + j], ch);
    }
    __syncthreads();
    for (int it0 = 0; it0 < nb * HALF; it0 += 256) {
      const int it = it0 + tid;
      const int jb = it / HALF, l = it % HALF;
      const int j = j0 + jb;
      float dot = 0.0f;
      if (jb < nb) {
        const float* lj = lat + jb * p.rmax;
        float klo = 0.0f, khi = 0.0f;
#pragma unroll 8
        for (int ch = 0; ch < r_g; ++ch) {
          klo = __builtin_fmaf(lj[ch], h2f(bk[ch * D + l]), klo);
          khi = __builtin_fmaf(lj[ch], h2f(bk[ch * D + l + HALF]), khi);
        }
        const float q_lo = p.q_bf16 ? __uint_as_float((uint32_t)qs[l] << 16) : h2f(qs[l]);
        const float q_hi = p.q_bf16 ? __uint_as_float((uint32_t)qs[l + HALF] << 16) : h2f(qs[l + HALF]);
        // angle t * theta^(-2l/D), reduced modulo 2 pi in fp64
        double ph = (double)c_t[j] * exp2(-(2.0 * l / D) * p.log2_theta);
        ph -= 6.283185307179586476925286766559 * floor(ph * 0.15915494309189533576888376337251);
        float sf, cf;
        sincosf((float)ph, &sf, &cf);
        dot = q_lo * (klo * cf - khi * sf) + q_hi * (khi * cf + klo * sf);
      }
      for (int o = HALF / 2; o > 0; o >>= 1) dot += __shfl_xor(dot, o);
      if (l == 0 && jb < nb)
        c_d[j] = __builtin_amdgcn_exp2f(dot * p.score_scale - M) - __builtin_amdgcn_exp2f(c_x[j] - M);
    }
    }
    __syncthreads();
    if (tid == 0) {
      float l2 = Lsum;
      for (int j = 0; j < n_sel; ++j) l2 += c_d[j];
      misc[2] = l2;
    }
    __syncthreads();
  } else if (tid == 0) {
    misc[2] = Lsum;
  }
  __syncthreads();
  const float inv_l = 1.0f / misc[2];
  auto merge_channel = [&](int r) {
    float acc = red4[r] + red4[p.rv + r] + red4[2 * p.rv + r] + red4[3 * p.rv + r];
    for (int j0 = 0; j0 < n_sel; j0 += 8) {   // eight candidates' loads in flight
      float vl[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) vl[u] = j0 + u < n_sel ? value_latent(p, b, c_t[j0 + u], r) : 0.0f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (j0 + u < n_sel) acc = __builtin_fmaf(c_d[j0 + u], vl[u], acc);
    }
    a[r] = acc * inv_l;
  };
  // (shallow form: the first rows of U_V, in flight while the rescored tokens'
  // value latents load)
  if constexpr (!DEEP) load_rows(rg, w0);
  for (int r = tid; r < p.rv; r += 256) merge_channel(r);
  __syncthreads();
  if (to_lat) {                 // absorbed output: the latents go to the product pass
    for (int r = tid; r < p.rv; r += 256) {
      const float x = a[r];
      const _Float16 h = (_Float16)x;
      p.lat[lat_row + r] = __builtin_bit_cast(uint16_t, h);
      p.lat[lat_lo + lat_row + r] = __builtin_bit_cast(uint16_t, (_Float16)(x - (float)h));
    }
    return;
  }
  // o = a . U_V^T restricted to KV head g's d columns (the reordering of Sec. 3.3):
  // thread (rg, j8) covers rows rg, rg + groups, .. and columns c_0 + 8*j8 ..+7
  float o[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  auto up_rows = [&](int r0, const u4 (&w8)[kUpRows]) {
#pragma unroll
    for (int k = 0; k < kUpRows; ++k) {
      const int r = r0 + k * groups;
      if (r < p.rv) {
        const _Float16* hw = reinterpret_cast<const _Float16*>(&w8[k]);
        const float ar = a[r];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] += ar * (float)hw[e];
      }
    }
  };
  up_rows(rg, w0);
  for (int r0 = rg + kUpRows * groups; r0 < p.rv; r0 += kUpRows * groups) {
    u4 w8[kUpRows];
    load_rows(r0, w8);
    up_rows(r0, w8);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[rg * Dc + 8 * j8 + e] = o[e];
  __syncthreads();
  if (tid < Dc) {
    float ov = 0.0f;
    for (int k = 0; k < groups; ++k) ov += red[k * Dc + tid];
    if (p.out_dtype == STARKV_DT_F32) {
      static_cast<float*>(p.out)[out_row + c_0 + tid] = ov;
    } else {
      uint16_t bits;
      if (p.out_dtype == STARKV_DT_BF16) {
        const uint32_t u = __float_as_uint(ov);
        bits = (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
        if ((u & 0x7F800000u) == 0x7F800000u) bits = (uint16_t)(u >> 16) | ((u & 0xFFFFu) ? 0x40 : 0);
      } else {
        bits = __builtin_bit_cast(uint16_t, (_Float16)ov);
      }
      static_cast<uint16_t*>(p.out)[out_row + c_0 + tid] = bits;
    }
  }
}
#endif  // SK_COMMON

// ---------------------------------------------------------------------- launchers
// The file is compiled once per (head_dim, cache precision) with SK_D and SK_QM
// set, producing the split-kernel instances for that pair, and once with
// SK_COMMON for the combine kernel and the dispatcher.
// Raises a kernel's dynamic LDS limit to 160 KiB once per device: `done` holds
// one bit per device index (indices past 63 set it on every launch).
static int allow_lds(const void* fn, std::atomic<uint64_t>& done) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  const uint64_t bit = dev < 64 ? 1ull << dev : 0;
  if (bit && (done.load(std::memory_order_acquire) & bit)) return 0;
  e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (e != hipSuccess) return (int)e;
  done.fetch_or(bit, std::memory_order_release);
  return 0;
}

#if defined(SK_D) && defined(SK_QM)
template <int D, int QM, int CT, int NTW>
static int launch_split_t(const DecodeParams& p, size_t lds, hipStream_t st) {
  auto k = decode_split_kernel<D, QM, CT, NTW>;
  static std::atomic<uint64_t> attr{0};
  if (const int e = allow_lds(reinterpret_cast<const void*>(k), attr)) return e;
  dim3 grid(p.dyn ? p.cap : p.n_split, p.dyn ? 1 : p.batch, p.n_hg);
  hipLaunchKernelGGL(k, grid, dim3(kThreads), lds, st, p);
  return (int)hipGetLastError();
}

template <int D, int QM, int CT>
static int dispatch_ntw(const DecodeParams& p, int ntw, size_t lds, hipStream_t st) {
  switch (ntw) {
    case 1: return launch_split_t<D, QM, CT, 1>(p, lds, st);
    case 2: return launch_split_t<D, QM, CT, 2>(p, lds, st);
    case 4: return launch_split_t<D, QM, CT, 4>(p, lds, st);
    case 8:
      if (CT <= 2) return launch_split_t<D, QM, CT, 8>(p, lds, st);
      break;
  }
  return (int)hipErrorInvalidValue;
}

#define SK_CAT2(a, b, c) launch_split_d##a##_q##b
#define SK_NAME(a, b) SK_CAT2(a, b, _)
int SK_NAME(SK_D, SK_QM)(const DecodeParams& p, int ct, int ntw, size_t lds, hipStream_t st) {
  switch (ct) {
    case 1: return dispatch_ntw<SK_D, SK_QM, 1>(p, ntw, lds, st);
    case 2: return dispatch_ntw<SK_D, SK_QM, 2>(p, ntw, lds, st);
    case 4: return dispatch_ntw<SK_D, SK_QM, 4>(p, ntw, lds, st);
  }
  return (int)hipErrorInvalidValue;
}
#endif

#ifdef SK_COMMON
#define SK_DECL(a, b) \
  int launch_split_d##a##_q##b(const DecodeParams& p, int ct, int ntw, size_t lds, hipStream_t st);
SK_DECL(64, 0) SK_DECL(64, 1) SK_DECL(64, 2) SK_DECL(64, 3)
SK_DECL(128, 0) SK_DECL(128, 1) SK_DECL(128, 2) SK_DECL(128, 3)

int split_lds_bytes(int frags, int nql, int head_dim, int ct, int raw_bytes, int v_ng,
                    int v_row_bytes) {
  return split_lds(frags, nql, head_dim, ct, raw_bytes, v_ng, kStepTokens * v_row_bytes).total;
}

int launch_decode_split_ntw(const DecodeParams& p, int head_dim, int qmode, int ct, int ntw,
                            size_t lds, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (head_dim == 128) {
    switch (qmode) {
      case STARKV_Q_F16: return launch_split_d128_q0(p, ct, ntw, lds, st);
      case STARKV_Q_INT4: return launch_split_d128_q1(p, ct, ntw, lds, st);
      case STARKV_Q_MIX8_4: return launch_split_d128_q2(p, ct, ntw, lds, st);
      case STARKV_Q_MIX4_3: return launch_split_d128_q3(p, ct, ntw, lds, st);
    }
  } else if (head_dim == 64) {
    switch (qmode) {
      case STARKV_Q_F16: return launch_split_d64_q0(p, ct, ntw, lds, st);
      case STARKV_Q_INT4: return launch_split_d64_q1(p, ct, ntw, lds, st);
      case STARKV_Q_MIX8_4: return launch_split_d64_q2(p, ct, ntw, lds, st);
      case STARKV_Q_MIX4_3: return launch_split_d64_q3(p, ct, ntw, lds, st);
    }
  }
  return (int)hipErrorInvalidValue;
}

// ---------------------------------------------------------------- fixed scratch
// Workspace of the no-allocation decode entry point: one array per device, kept
// until the process ends.  Its device address comes from hipGetSymbolAddress,
// taken once per device with that device current; host code never passes the
// array's name to a kernel (in host code the name is a host-side stand-in).
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

int scratch_address(void** out) {
  constexpr int kMaxDevices = 64;
  static std::atomic<void*> addr[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
  void* p = addr[dev].load(std::memory_order_acquire);
  if (!p) {
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return (int)e;
    if (!p) return (int)hipErrorInvalidSymbol;
    addr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return 0;
}

int launch_decode_combine(const CombineParams& p, void* stream) {
  if (p.n_split > kCombineMaxSplits) return (int)hipErrorInvalidValue;
  // the shared region: the merge phase (split sums, rescoring latents, B_k
  // block) or the up-projection's 256 / (D/8) rows of D partial sums
  const size_t merge = (size_t)4 * p.rv + (size_t)kRescoreBatch * p.rmax + (size_t)p.rmax * p.head_dim / 2;
  if (p.col_split != 1 && (p.col_split != 2 || p.lat)) return (int)hipErrorInvalidValue;
  const int dc = p.head_dim / p.col_split;
  const size_t upproj = (size_t)256 / (dc / 8) * dc;
  const size_t lds = ((size_t)combine_head_floats(p.rv) + (merge > upproj ? merge : upproj)) *
                     sizeof(float);
  dim3 grid(p.n_q, p.batch, p.col_split);
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if ((int64_t)p.n_q * p.batch * p.col_split <= 256) {
    static std::atomic<uint64_t> attr{0};
    if (const int e = allow_lds(reinterpret_cast<const void*>(decode_combine_kernel<true>), attr)) return e;
    hipLaunchKernelGGL(decode_combine_kernel<true>, grid, dim3(256), lds, st, p);
  } else {
    static std::atomic<uint64_t> attr{0};
    if (const int e = allow_lds(reinterpret_cast<const void*>(decode_combine_kernel<false>), attr)) return e;
    hipLaunchKernelGGL(decode_combine_kernel<false>, grid, dim3(256), lds, st, p);
  }
  return (int)hipGetLastError();
}
#endif

}  // namespace starkv
