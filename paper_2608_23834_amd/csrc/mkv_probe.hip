// Streaming-read probe: reads a device buffer once with 16-byte loads, four
// in flight per lane, and folds it into one word per workgroup.  It measures
// the HBM read bandwidth a kernel that touches each byte once can reach on
// this device, the ceiling the decode scan is compared against.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mkv_internal.h"
#include "../../include/minima_kv.h"

namespace mkv {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4* __restrict__ src, int64_t n_vec,
                                                          uint32_t* __restrict__ sink) {
  constexpr int U = 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (U - 1) * stride < n_vec; i += U * stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  for (; i < n_vec; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(src + i);
    acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  // fold the workgroup's words so the loads stay live; one store per workgroup
  for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o, 64);
  __shared__ uint32_t s[4];
  if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = s[0] ^ s[1] ^ s[2] ^ s[3];
}

hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, int n_wg, hipStream_t s) {
  hipLaunchKernelGGL(stream_read_kernel, dim3(n_wg), dim3(256), 0, s,
                     reinterpret_cast<const u32x4*>(buf), (int64_t)(bytes / 16), sink);
  return hipGetLastError();
}

}  // namespace mkv
