// starkv_append kernels (gfx950).
//
// downproj: latents = x . A_all (Sec. 3.2: K' = x (Sigma V)_K per head, V' =
//   x (Sigma V)_V), bf16 operands on v_mfma_f32_16x16x32_bf16, fp32 partial sums
//   per k-split, then a fixed-order reduction rounded to fp16.
// pack: per-token group quantization of every latent block into the cache
//   (Sec. 4.4: outlier block at 8 bits, inlier block at 4 bits).  The scale is
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

// ------------------------------------------------------------------ pack kernel
// One thread per (sequence b, 32-token block touched, chunk q of that block,
// (latent block, group) item).  The thread handles the eight tokens of value
// chunk q (4q..4q+3, 16+4q..16+4q+3), so every 32-bit value word is owned by
// exactly one thread; tokens outside [pos, pos+n_new) keep their old bits.

__global__ __launch_bounds__(256) void pack_kernel(AppendParams p) {
  const int item = blockIdx.x * blockDim.x + threadIdx.x;
  if (item >= p.n_items) return;
  const int kq = blockIdx.y & 3;
  const int bj = blockIdx.y >> 2;           // block index within the touched range
  const int b = blockIdx.z;
  const int pos = p.pos[b];
  const int blk = (pos >= 0 ? pos / 32 : -((31 - pos) / 32)) + bj;
  const int blk_end = (pos + p.n_new - 1 >= 0) ? (pos + p.n_new - 1) / 32 : -1;
  if (blk > blk_end || blk < 0) return;
  const int bl = p.item_block[item], gi = p.item_group[item];
  const int r = p.rank[bl], ro = p.ro[bl];
  const bool is_v = (bl == p.n_kv);
  const int qm = p.qmode;
  // group channel range and bit width
  int c0, n, bits;
  if (qm == STARKV_Q_F16) {
    c0 = 32 * gi; n = min(32, r - c0); bits = 16;
  } else {
    const int ng8 = (ro + 31) / 32;
    if (gi < ng8) { c0 = 32 * gi; n = min(32, ro - c0); bits = 8; }
    else { c0 = ro + 32 * (gi - ng8); n = min(32, r - c0); bits = 4; }
  }
  uint8_t* code_plane = p.cache + p.code_off[bl];
  uint8_t* meta_plane = p.cache + p.meta_off[bl];
  const int rb = p.row_bytes[bl];
  const int ngr = p.ng[bl];
  uint32_t words[32];                        // value 4-bit chunk words, one per channel
  bool have_words = false;
  const int64_t vblk = (int64_t)b * (p.cap_pad / 32) + blk;
  uint8_t* vblock = code_plane + vblk * 32 * rb;
  const int ri = r - ro;

  for (int slot = 0; slot < 8; ++slot) {
    const int u = (slot < 4) ? (4 * kq + slot) : (16 + 4 * kq + slot - 4);
    const int t = blk * 32 + u;
    if (t < pos || t >= pos + p.n_new || t >= p.capacity) continue;
    const uint16_t* x = p.lat + ((int64_t)b * p.n_new + (t - pos)) * p.width + p.lat_off[bl] + c0;
    if (!is_v) {
      const int64_t kblk = (int64_t)b * (p.cap_pad / 16) + t / 16;
      const int tau = t % 16;
      uint8_t* kb = code_plane + kblk * 16 * rb;
      if (bits == 16) {
        for (int i = 0; i < n; ++i) {
          const int c = c0 + i;
          *reinterpret_cast<uint16_t*>(kb + (c / 8) * 256 + tau * 16 + (c % 8) * 2) = x[i];
        }
        continue;
      }
      const GroupQ g = group_params(x, n, bits);
      const int n8 = ro / 8;
      for (int i = 0; i < n; i += 8) {         // one chunk of 8 channels at a time
        const int c = c0 + i, ch = c / 8;
        if (bits == 8) {
          uint32_t lo = 0, hi = 0;
          for (int k = 0; k < 4; ++k) lo |= group_code(g, x[i + k]) << (8 * k);
          for (int k = 0; k < 4; ++k) hi |= group_code(g, x[i + 4 + k]) << (8 * k);
          uint32_t* dst = reinterpret_cast<uint32_t*>(kb + ch * 128 + tau * 8);
          dst[0] = lo;
          dst[1] = hi;
        } else {
          uint32_t wv = 0;
          for (int k = 0; k < 8; ++k) wv |= group_code(g, x[i + k]) << (4 * k);
          *reinterpret_cast<uint32_t*>(kb + n8 * 128 + (ch - n8) * 64 + tau * 4) = wv;
        }
      }
      uint16_t* m = reinterpret_cast<uint16_t*>(meta_plane + (kblk * ngr + gi) * 64 + tau * 4);
      m[0] = g.s;
      m[1] = g.z;
    } else {
      if (bits == 16) {
        for (int i = 0; i < n; ++i) {
          const int c = c0 + i;
          *reinterpret_cast<uint16_t*>(vblock + ((int64_t)c * 4 + kq) * 16 + slot * 2) = x[i];
        }
        continue;
      }
      const GroupQ g = group_params(x, n, bits);
      if (bits == 8) {
        for (int i = 0; i < n; ++i) {
          const int c = c0 + i;
          vblock[((int64_t)c * 4 + kq) * 8 + slot] = (uint8_t)group_code(g, x[i]);
        }
      } else {
        if (!have_words) {
          for (int i = 0; i < n; ++i)
            words[i] = *reinterpret_cast<const uint32_t*>(
                vblock + 32 * ro + ((int64_t)(c0 - ro + i) * 4 + kq) * 4);
          have_words = true;
        }
        // slot 2k -> bits 4k..4k+3, slot 2k+1 -> bits 16+4k..16+4k+3
        const int sh = (slot % 2 == 0) ? 4 * (slot / 2) : 16 + 4 * (slot / 2);
        for (int i = 0; i < n; ++i)
          words[i] = (words[i] & ~(0xFu << sh)) | (group_code(g, x[i]) << sh);
      }
      uint16_t* m = reinterpret_cast<uint16_t*>(meta_plane +
                                                (vblk * ngr + gi) * 128 + kq * 32 + slot * 2);
      m[0] = g.s;
      m[8] = g.z;
    }
  }
  if (have_words) {
    for (int i = 0; i < n; ++i)
      *reinterpret_cast<uint32_t*>(vblock + 32 * ro + ((int64_t)(c0 - ro + i) * 4 + kq) * 4) =
          words[i];
  }
}

// ------------------------------------------------------------------ down-projection
constexpr int BM = 64, BN = 64, BK = 32;

__global__ __launch_bounds__(256) void downproj_kernel(DownprojParams p) {
  __shared__ __align__(16) __bf16 xs[BM][BK + 8];
  __shared__ __align__(16) __bf16 as[BN][BK + 8];    // transposed A tile: [n][k]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM, ks = blockIdx.z;
  const int k_lo = ks * p.k_chunk;
  const int k_hi = min(p.k, k_lo + p.k_chunk);
  const int wm = (w >> 1) * 32, wn = (w & 1) * 32;
  f4 acc[2][2];
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j) acc[i][j] = (f4){0, 0, 0, 0};
  for (int k0 = k_lo; k0 < k_hi; k0 += BK) {
    // x tile: 64 rows x 32 k, 8 elements per thread
    {
      const int r = tid / 4, kk = (tid % 4) * 8;
      const int m = m0 + r;
      u4 v = (u4){0, 0, 0, 0};
      if (m < p.m && k0 + kk + 8 <= k_hi) {
        v = *reinterpret_cast<const u4*>(p.x + (int64_t)m * p.k + k0 + kk);
      } else if (m < p.m) {
        uint16_t tmp[8];
        for (int e = 0; e < 8; ++e)
          tmp[e] = (k0 + kk + e < k_hi) ? p.x[(int64_t)m * p.k + k0 + kk + e] : (uint16_t)0;
        v = *reinterpret_cast<u4*>(tmp);
      }
      *reinterpret_cast<u4*>(&xs[r][kk]) = v;
    }
    // A tile: 32 k x 64 n, stored transposed
    {
      const int kr = tid / 8, nn = (tid % 8) * 8;
      const int k = k0 + kr;
      uint16_t tmp[8];
      for (int e = 0; e < 8; ++e) {
        const int n = n0 + nn + e;
        tmp[e] = (k < k_hi && n < p.n) ? p.a[(int64_t)k * p.n + n] : (uint16_t)0;
      }
      for (int e = 0; e < 8; ++e) as[nn + e][kr] = __builtin_bit_cast(__bf16, tmp[e]);
    }
    __syncthreads();
    const int row = lane & 15, kq = lane >> 4;
    b8 af[2], bf[2];
    for (int i = 0; i < 2; ++i) af[i] = *reinterpret_cast<const b8*>(&xs[wm + 16 * i + row][8 * kq]);
    for (int j = 0; j < 2; ++j) bf[j] = *reinterpret_cast<const b8*>(&as[wn + 16 * j + row][8 * kq]);
    for (int i = 0; i < 2; ++i)
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
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

__global__ __launch_bounds__(256) void downproj_reduce_kernel(DownprojParams p) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t mn = (int64_t)p.m * p.n;
  if (i >= mn) return;
  float s = 0.0f;
  for (int k = 0; k < p.k_split; ++k) s += p.partial[k * mn + i];
  p.lat[i] = __builtin_bit_cast(uint16_t, (_Float16)s);
}

// ------------------------------------------------------------------ launchers
int launch_append_pack(const AppendParams& p, void* stream) {
  const int nblk = p.n_new / 32 + 2;          // 32-token blocks a range of n_new rows can touch
  dim3 grid((p.n_items + 63) / 64, nblk * 4, p.batch);
  hipLaunchKernelGGL(pack_kernel, grid, dim3(64), 0, static_cast<hipStream_t>(stream), p);
  return (int)hipGetLastError();
}

int launch_downproj(const DownprojParams& p, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  dim3 grid((p.n + BN - 1) / BN, (p.m + BM - 1) / BM, p.k_split);
  hipLaunchKernelGGL(downproj_kernel, grid, dim3(256), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  const int64_t mn = (int64_t)p.m * p.n;
  hipLaunchKernelGGL(downproj_reduce_kernel, dim3((unsigned)((mn + 255) / 256)), dim3(256), 0, st,
                     p);
  return (int)hipGetLastError();
}

}  // namespace starkv
