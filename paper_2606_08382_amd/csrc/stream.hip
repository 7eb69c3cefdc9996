// Plain HBM read stream: the measured ceiling that the decode kernels' latent
// stream is reported against.  Every lane keeps sixteen 16-byte loads in flight
// (grid-stride), folds what it reads with XOR, and each wave writes one word,
// so the loads cannot be removed and the writes are negligible.  Four loads in
// flight per lane read 1 GiB at 5.3 TB/s, eight at 6.2-6.3 and sixteen at
// 6.3-6.4 TB/s: the bytes in flight per compute unit set the rate.
#include <hip/hip_runtime.h>

#include "starkv_internal.h"

namespace starkv {

typedef uint32_t u4s __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void read_stream_kernel(const u4s* __restrict__ src,
                                                          int64_t n_vec, uint32_t* sink) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  constexpr int U = 16;
  u4s acc[U];
#pragma unroll
  for (int u = 0; u < U; ++u) acc[u] = (u4s){0, 0, 0, 0};
  for (; i + (U - 1) * stride < n_vec; i += U * stride) {
#pragma unroll
    for (int u = 0; u < U; ++u) acc[u] ^= src[i + u * stride];
  }
  for (; i < n_vec; i += stride) acc[0] ^= src[i];
  u4s x = acc[0];
#pragma unroll
  for (int u = 1; u < U; ++u) x ^= acc[u];
  uint32_t v = x.x ^ x.y ^ x.z ^ x.w;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v ^= __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) sink[(blockIdx.x * 256 + threadIdx.x) >> 6] = v;
}

int launch_read_stream(const void* src, int64_t bytes, uint32_t* sink, int workgroups,
                       void* stream) {
  hipLaunchKernelGGL(read_stream_kernel, dim3(workgroups), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u4s*>(src), bytes / 16,
                     sink);
  return (int)hipGetLastError();
}

}  // namespace starkv
