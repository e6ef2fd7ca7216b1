// Bandwidth probes: a plain copy (byte-counter calibration) and a streaming read.
#include <hip/hip_runtime.h>

#include "treepo.h"
#include "treepo_bench.h"

namespace {

constexpr int kThreads = 256;
constexpr unsigned kGrid = 4096;

__global__ __launch_bounds__(kThreads) void copy_kernel(uint4* __restrict__ dst, const uint4* __restrict__ src,
                                                        int64_t n) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kThreads)
    dst[i] = src[i];
}

__global__ __launch_bounds__(kThreads) void read_kernel(const uint4* __restrict__ src, int64_t n,
                                                        float* __restrict__ sink) {
  uint32_t acc = 0;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kThreads) {
    const uint4 v = src[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  __shared__ uint32_t red[kThreads];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if (static_cast<int>(threadIdx.x) < s) red[threadIdx.x] ^= red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) sink[blockIdx.x] = static_cast<float>(red[0] & 0xFFFF);
}

}  // namespace

extern "C" int32_t treepo_bench_copy(void* dst, const void* src, size_t bytes, hipStream_t stream) {
  if (!dst || !src || bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) % 16)
    return TREEPO_EINVAL;
  copy_kernel<<<kGrid, kThreads, 0, stream>>>(static_cast<uint4*>(dst), static_cast<const uint4*>(src),
                                              static_cast<int64_t>(bytes / 16));
  return hipGetLastError() == hipSuccess ? TREEPO_OK : TREEPO_EHIP;
}

extern "C" int32_t treepo_bench_read(const void* src, size_t bytes, float* sink, hipStream_t stream) {
  if (!src || !sink || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(src) % 16) return TREEPO_EINVAL;
  read_kernel<<<kGrid, kThreads, 0, stream>>>(static_cast<const uint4*>(src), static_cast<int64_t>(bytes / 16), sink);
  return hipGetLastError() == hipSuccess ? TREEPO_OK : TREEPO_EHIP;
}
