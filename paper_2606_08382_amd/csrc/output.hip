// Attention-block output with the value up-projection absorbed into the
// output projection (gfx950).
//
// Sec. 3.3 (weight absorption): o_i W_out,i^T = (a_i / l_i) U_V^T W_out,i^T, and
// W'_out,i = W_out,i U_V,g(i) is formed offline, so the decode step never
// up-projects the value latent: y_b = sum_i W'_out,i (a_i / l_i).  With the
// heads' W'_out side by side this is one product y = lat . W_abs^T of the
// normalized latents lat [B][H_q * r_v] and W_abs [d_out][H_q * r_v].
//
// The product is bound by the HBM stream of W_abs (2 B per element, read once);
// each element is used B times.  It runs on v_mfma_f32_16x16x32_f16: the latent
// rows are the A operand (16 sequences per tile), W_abs rows the B operand (16
// output columns per tile).  The combine pass hands the fp32 latents over as two
// fp16 parts, hi = fp16(x) and lo = fp16(x - hi); both products are exact in the
// fp32 accumulator, so the latents enter with about 22 bits.
#include <hip/hip_runtime.h>

#include "starkv_internal.h"

namespace starkv {

#ifndef ABS_SK
#define ABS_SK 512
#define ABS_NB 8
#endif

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int kOutWaves = 16;      // waves per workgroup, each a slice of the k blocks
constexpr int kOutCols = 16;       // output columns per workgroup
constexpr int kOutRows = 64;       // sequences per workgroup (grid.y covers more)

__device__ __forceinline__ f4 mfma16(u4 a, u4 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a),
                                                __builtin_bit_cast(h8, b), c, 0, 0, 0);
}

// Workgroup (16 output columns, up to 64 sequences); wave w takes the k blocks
// (32 latent channels) w, w + 16, .., so at any time the waves read adjacent
// 64-byte pieces of the same 16 rows of W_abs.  NB = 16-row tiles of sequences.
template <int NB>
__global__ __launch_bounds__(kOutWaves * 64) void absorbed_out_kernel(AbsorbParams p) {
  constexpr int U = 8 / NB;                  // k blocks per round of loads
  __shared__ float red[kOutWaves][NB * 256];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n0 = blockIdx.x * kOutCols, b0 = blockIdx.y * kOutRows;
  const int K = p.k, B = p.batch;
  const int nkb = (K + 31) / 32;
  const int ksub = 8 * (lane >> 4);          // the lane's 8 channels inside a k block
  // B operand: row n of W_abs (rows past d_out read the last row; never stored)
  const uint16_t* wrow = p.w + (int64_t)min(n0 + (lane & 15), p.n_out - 1) * K + ksub;
  // A operand: sequence b0 + 16 t + (lane & 15), hi parts then lo parts
  const uint16_t* hi = p.lat + ksub;
  const uint16_t* lo = p.lat + (int64_t)B * K + ksub;
  int brow[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t) brow[t] = b0 + 16 * t + (lane & 15);
  f4 acc[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t) acc[t] = (f4){0, 0, 0, 0};
  for (int kb0 = w; kb0 < nkb; kb0 += kOutWaves * U) {
    u4 wf[U], ah[U][NB], al[U][NB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb0 + kOutWaves * u;
      const bool ok = kb < nkb && kb * 32 + ksub < K;   // K is a multiple of 8
      wf[u] = ok ? *reinterpret_cast<const u4*>(wrow + kb * 32) : (u4){0, 0, 0, 0};
#pragma unroll
      for (int t = 0; t < NB; ++t) {
        const bool okb = ok && brow[t] < B;
        const int64_t o = (int64_t)brow[t] * K + kb * 32;
        ah[u][t] = okb ? *reinterpret_cast<const u4*>(hi + o) : (u4){0, 0, 0, 0};
        al[u][t] = okb ? *reinterpret_cast<const u4*>(lo + o) : (u4){0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < NB; ++t) {
        acc[t] = mfma16(ah[u][t], wf[u], acc[t]);
        acc[t] = mfma16(al[u][t], wf[u], acc[t]);
      }
  }
  // lane holds rows 4*(lane/16)+e (sequences) of column lane%16 (outputs)
#pragma unroll
  for (int t = 0; t < NB; ++t)
#pragma unroll
    for (int e = 0; e < 4; ++e) red[w][(t * 4 + e) * 64 + lane] = acc[t][e];
  __syncthreads();
  for (int idx = threadIdx.x; idx < NB * 256; idx += kOutWaves * 64) {
    float s = 0.0f;
#pragma unroll
    for (int ww = 0; ww < kOutWaves; ++ww) s += red[ww][idx];
    const int t = idx >> 8, e = (idx >> 6) & 3, l = idx & 63;
    const int b = b0 + 16 * t + 4 * (l >> 4) + e, n = n0 + (l & 15);
    if (b >= B || n >= p.n_out) continue;
    const int64_t o = (int64_t)b * p.n_out + n;
    if (p.out_dtype == STARKV_DT_F32) {
      static_cast<float*>(p.out)[o] = s;
    } else if (p.out_dtype == STARKV_DT_BF16) {
      const uint32_t u = __float_as_uint(s);
      uint16_t bits = (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
      if ((u & 0x7F800000u) == 0x7F800000u) bits = (uint16_t)(u >> 16) | ((u & 0xFFFFu) ? 0x40 : 0);
      static_cast<uint16_t*>(p.out)[o] = bits;
    } else {
      static_cast<uint16_t*>(p.out)[o] = __builtin_bit_cast(uint16_t, (_Float16)s);
    }
  }
}

// Up to 16 sequences with K a multiple of NB * SK.  A load of the kernel
// above covers 64 bytes in each of 16 rows of W_abs that lie K * 2 bytes
// apart; here the workgroup's 16 rows go through LDS in stages of SK
// channels, every row copied as contiguous 1 KiB runs (global_load_lds, 16
// bytes per lane), and the MFMA B operands are read from LDS.  Rows are padded
// to SK * 2 + 16 bytes, so that the 16 lanes of a fragment read start in 16
// distinct groups of four banks.  NB buffers, NB - 1 stages in flight (one
// workgroup per CU).  A stage's group of loads is the wave's SK / 512 copies
// and its latent fragments (k blocks w + 16 i of the stage, hi and lo), so
// that waiting for a stage is a vmcnt of 3 SK / 512 per later stage.  The
// barrier is a bare s_barrier after the LDS reads have landed: the waits for
// the copies are the explicit vmcnts, and a __syncthreads() would also wait
// for the stages still in flight.
template <int V>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(V >= 0 && V < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (V & 15) | ((V >> 4) << 14));
}

constexpr int SK = ABS_SK, NB = ABS_NB;   // stage channels, LDS buffers

__global__ __launch_bounds__(kOutWaves * 64) void absorbed_out_lds_kernel(AbsorbParams p) {
  static_assert(kOutWaves == 16 && kOutCols == 16 && SK % 512 == 0 && SK <= 1024,
                "one or two 1 KiB copies and k blocks per wave and stage");
  constexpr int CPW = SK / 512;              // copies and k blocks per wave and stage
  constexpr int OPS = 3 * CPW;               // loads per wave and stage
  constexpr int ROW = SK * 2 + 16;           // bytes per staged row
  constexpr int SB = kOutCols * ROW;         // bytes per stage
  constexpr int AHEAD = NB - 1;              // stages in flight
  __shared__ __align__(16) uint8_t osm[NB * SB];
  __shared__ float red[kOutWaves][256];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n0 = blockIdx.x * kOutCols;
  const int K = p.k, nst = K / SK;           // a multiple of NB
  const int ksub = 8 * (lane >> 4);
  // copy i of a stage: j = w + 16 i, row j / CPW, 1 KiB run j % CPW (rows past
  // d_out copy the last row; never stored)
  const uint16_t* wsrc[CPW];
  int wd[CPW];
#pragma unroll
  for (int i = 0; i < CPW; ++i) {
    const int j = w + 16 * i, r = j / CPW, run = j % CPW;
    wsrc[i] = p.w + (int64_t)min(n0 + r, p.n_out - 1) * K + 512 * run + 8 * lane;
    wd[i] = r * ROW + 1024 * run;
  }
  // A operand: sequence lane & 15 (rows past the batch repeat the last
  // sequence; their outputs are never stored)
  const int brow = min(lane & 15, p.batch - 1);
  const uint16_t* hi = p.lat + (int64_t)brow * K + ksub + 32 * w;
  const uint16_t* lo = hi + (int64_t)p.batch * K;
  // the fragment reads are written out: the compiler would put a wait for every
  // copy in flight (vmcnt(0)) in front of an LDS read it sees
  typedef __attribute__((address_space(3))) uint8_t lds_u8;
  const uint32_t sw_lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_u8*)osm)) +
                          (lane & 15) * ROW + 2 * ksub + 64 * w;
  u4 lat[NB][2 * CPW];
  f4 acc = (f4){0, 0, 0, 0};
  auto issue = [&](int st, u4(&l)[2 * CPW]) {
    uint8_t* dst = osm + (st % NB) * SB;
    const int64_t c = (int64_t)st * SK;
#pragma unroll
    for (int i = 0; i < CPW; ++i) __builtin_amdgcn_global_load_lds(wsrc[i] + c, dst + wd[i], 16, 0, 0);
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      l[2 * i] = *reinterpret_cast<const u4*>(hi + c + 512 * i);
      l[2 * i + 1] = *reinterpret_cast<const u4*>(lo + c + 512 * i);
    }
  };
  // stage st (buffer u = st % NB) with `later` stages still in flight after
  // it; the fragments are read before the next copies go out, which then take
  // buffer (u + AHEAD) % NB, the one that held stage st - 1
  // `later` is a constant once the loops below are unrolled: the switch folds
  auto wait_later = [](int later) {
    static_assert(AHEAD <= 8, "cases below");
    switch (later) {
      case 0: wait_vmcnt<0>(); break;
      case 1: wait_vmcnt<OPS>(); break;
      case 2: wait_vmcnt<2 * OPS>(); break;
      case 3: wait_vmcnt<3 * OPS>(); break;
      case 4: wait_vmcnt<4 * OPS>(); break;
      case 5: wait_vmcnt<5 * OPS>(); break;
      case 6: wait_vmcnt<6 * OPS>(); break;
      default: wait_vmcnt<7 * OPS>(); break;
    }
  };
  auto step = [&](int later, int u, int st, bool more) {
    wait_later(later);
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    u4 bf[CPW];
    if constexpr (CPW == 2) {
      asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %2 offset:1024"
                   : "=v"(bf[0]), "=v"(bf[1]) : "v"(sw_lds + u * SB) : "memory");
    } else {
      asm volatile("ds_read_b128 %0, %1" : "=v"(bf[0]) : "v"(sw_lds + u * SB) : "memory");
    }
    if (more) issue(st + AHEAD, lat[(u + AHEAD) % NB]);
    if constexpr (CPW == 2) asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(bf[0]), "+v"(bf[1]) :: "memory");
    else asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(bf[0]) :: "memory");
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      acc = mfma16(lat[u][2 * i], bf[i], acc);
      acc = mfma16(lat[u][2 * i + 1], bf[i], acc);
    }
  };
#pragma unroll
  for (int st = 0; st < AHEAD; ++st) issue(st, lat[st]);
  int s0 = 0;
  for (; s0 < nst - NB; s0 += NB) {
#pragma unroll
    for (int u = 0; u < NB; ++u) step(AHEAD - 1, u, s0 + u, true);
  }
  // the last NB stages: stage s0 + u has min(AHEAD - 1, NB - 1 - u) later
  // stages in flight, and only the first still issues one
#pragma unroll
  for (int u = 0; u < NB; ++u) step(min(AHEAD - 1, NB - 1 - u), u, s0 + u, u == 0);
  // lane holds rows 4*(lane/16)+e (sequences) of column lane%16 (outputs)
#pragma unroll
  for (int e = 0; e < 4; ++e) red[w][e * 64 + lane] = acc[e];
  __syncthreads();
  for (int idx = threadIdx.x; idx < 256; idx += kOutWaves * 64) {
    float s = 0.0f;
#pragma unroll
    for (int ww = 0; ww < kOutWaves; ++ww) s += red[ww][idx];
    const int e = (idx >> 6) & 3, l = idx & 63;
    const int b = 4 * (l >> 4) + e, n = n0 + (l & 15);
    if (b >= p.batch || n >= p.n_out) continue;
    const int64_t o = (int64_t)b * p.n_out + n;
    if (p.out_dtype == STARKV_DT_F32) {
      static_cast<float*>(p.out)[o] = s;
    } else if (p.out_dtype == STARKV_DT_BF16) {
      const uint32_t u = __float_as_uint(s);
      uint16_t bits = (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
      if ((u & 0x7F800000u) == 0x7F800000u) bits = (uint16_t)(u >> 16) | ((u & 0xFFFFu) ? 0x40 : 0);
      static_cast<uint16_t*>(p.out)[o] = bits;
    } else {
      static_cast<uint16_t*>(p.out)[o] = __builtin_bit_cast(uint16_t, (_Float16)s);
    }
  }
}

int launch_absorbed_out(const AbsorbParams& p, void* stream) {
  if (p.n_out < 1 || p.k < 8 || p.k % 8 || p.batch < 1) return (int)hipErrorInvalidValue;
  dim3 grid((p.n_out + kOutCols - 1) / kOutCols, (p.batch + kOutRows - 1) / kOutRows);
  dim3 block(kOutWaves * 64);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (p.batch <= 16 && p.k % (ABS_NB * ABS_SK) == 0)
    hipLaunchKernelGGL(absorbed_out_lds_kernel, dim3(grid.x), block, 0, st, p);
  else if (p.batch <= 16) hipLaunchKernelGGL(absorbed_out_kernel<1>, grid, block, 0, st, p);
  else if (p.batch <= 32) hipLaunchKernelGGL(absorbed_out_kernel<2>, grid, block, 0, st, p);
  else hipLaunchKernelGGL(absorbed_out_kernel<4>, grid, block, 0, st, p);
  return (int)hipGetLastError();
}

}  // namespace starkv
