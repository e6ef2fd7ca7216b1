// Bandwidth probes: a plain copy (byte-counter calibration) and a streaming
// read; and a probe of how matrix-core and vector-ALU work share a SIMD.
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

// Streaming reads with the staging pattern of the decode kernels: 16 KiB
// chunks moved with 16-byte global->LDS loads into a ring of four LDS buffers,
// three chunks in flight, one workgroup barrier per chunk.  `blocked` selects
// whether each workgroup streams one contiguous share (as a decode work item
// does) or takes chunks grid-stride.
constexpr int kChunk = 16384;

template <bool NT>
__device__ __forceinline__ void lds_load16(const void* g, uint32_t lds) {
  if (NT)
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                 :: "v"(g), "s"(lds) : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(g), "s"(lds) : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void landed_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(N) : "memory");
}

template <bool NT>
__global__ __launch_bounds__(kThreads) void stream_lds_kernel(const char* __restrict__ src, int64_t nchunks,
                                                              int32_t blocked, float* __restrict__ sink) {
  __shared__ __attribute__((aligned(1024))) char buf[4][kChunk];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t G = gridDim.x;
  const int64_t per = nchunks / G;
  const int64_t first = blocked ? blockIdx.x * per : blockIdx.x;
  const int64_t step = blocked ? 1 : G;
  const int64_t count = blocked ? per : (nchunks - blockIdx.x + G - 1) / G;
  const uint32_t base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(
      (const __attribute__((address_space(3))) char*)&buf[0][0]));
  auto issue = [&](int64_t i) {
    const char* g = src + (first + i * step) * kChunk;
    const uint32_t b = base + static_cast<uint32_t>(i & 3) * kChunk;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int slot = wave * 4 + j;
      lds_load16<NT>(g + slot * 1024 + lane * 16, __builtin_amdgcn_readfirstlane(b + slot * 1024));
    }
  };
  for (int64_t p = 0; p < 3 && p < count; ++p) issue(p);
  uint32_t acc = 0;
  for (int64_t i = 0; i < count; ++i) {
    const int64_t ahead = count - 1 - i;
    if (ahead >= 2)
      landed_barrier<8>();
    else if (ahead == 1)
      landed_barrier<4>();
    else
      landed_barrier<0>();
    if (i + 3 < count) issue(i + 3);
    acc ^= reinterpret_cast<const uint32_t*>(buf[i & 3])[threadIdx.x];
  }
  if (threadIdx.x == 0) sink[blockIdx.x] = static_cast<float>(acc & 0xFFFF);
}

// Each workgroup streams one contiguous share with 16-byte register loads.
__global__ __launch_bounds__(kThreads) void stream_reg_kernel(const uint4* __restrict__ src, int64_t n16_per_wg,
                                                              float* __restrict__ sink) {
  const uint4* p = src + blockIdx.x * n16_per_wg;
  uint32_t acc = 0;
#pragma unroll 4
  for (int64_t i = threadIdx.x; i < n16_per_wg; i += kThreads) {
    const uint4 v = p[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (threadIdx.x == 0) sink[blockIdx.x] = static_cast<float>(acc & 0xFFFF);
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// One workgroup; every wave runs `iters` rounds of eight independent
// v_mfma_f32_16x16x32_bf16 (MF) and/or 24 independent FMAs (VA), issued as
// one MFMA then three FMAs, and stores its own clock delta (s_memtime).
template <bool MF, bool VA>
__global__ __launch_bounds__(1024) void overlap_kernel(float* __restrict__ sink, uint64_t* __restrict__ cycles,
                                                       int iters) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = static_cast<__bf16>(0.001f * (lane + i));
    b[i] = static_cast<__bf16>(0.002f * (lane - i));
  }
  f32x4 acc[8];
  for (int j = 0; j < 8; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float x[16];
  for (int j = 0; j < 16; ++j) x[j] = 0.01f * (lane + j);
  const uint64_t t0 = __builtin_amdgcn_s_memtime();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (MF) acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
      if (VA) {
#pragma unroll
        for (int v = 0; v < 3; ++v) x[(3 * j + v) & 15] = fmaf(x[(3 * j + v) & 15], 0.999f, 0.001f);
      }
      if (MF) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (VA) __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
    }
  }
  const uint64_t t1 = __builtin_amdgcn_s_memtime();
  float sum = 0.f;
  for (int j = 0; j < 8; ++j) sum += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
  for (int j = 0; j < 16; ++j) sum += x[j];
  sink[threadIdx.x] = sum;
  if (lane == 0) cycles[threadIdx.x >> 6] = t1 - t0;
}

}  // namespace

extern "C" int32_t treepo_bench_overlap(int32_t mode, int32_t waves_per_simd, int32_t iters, float* sink,
                                        uint64_t* cycles, hipStream_t stream) {
  if (!sink || !cycles || mode < 0 || mode > 2 || waves_per_simd < 1 || waves_per_simd > 4 || iters < 1)
    return TREEPO_EINVAL;
  const dim3 block(256 * waves_per_simd);
  if (mode == 0)
    overlap_kernel<true, false><<<1, block, 0, stream>>>(sink, cycles, iters);
  else if (mode == 1)
    overlap_kernel<false, true><<<1, block, 0, stream>>>(sink, cycles, iters);
  else
    overlap_kernel<true, true><<<1, block, 0, stream>>>(sink, cycles, iters);
  return hipGetLastError() == hipSuccess ? TREEPO_OK : TREEPO_EHIP;
}

extern "C" int32_t treepo_bench_stream(const void* src, size_t bytes, float* sink, int32_t mode,
                                       int32_t workgroups, hipStream_t stream) {
  if (!src || !sink || workgroups < 1 || workgroups > 4096 || reinterpret_cast<uintptr_t>(src) % 16 ||
      mode < 0 || mode > 3)
    return TREEPO_EINVAL;
  if (bytes % (static_cast<size_t>(kChunk) * workgroups) != 0) return TREEPO_EINVAL;
  const int64_t nchunks = static_cast<int64_t>(bytes / kChunk);
  if (mode == 2)
    stream_reg_kernel<<<workgroups, kThreads, 0, stream>>>(static_cast<const uint4*>(src),
                                                           static_cast<int64_t>(bytes / 16 / workgroups), sink);
  else if (mode == 3)
    stream_lds_kernel<true><<<workgroups, kThreads, 0, stream>>>(static_cast<const char*>(src), nchunks, 1, sink);
  else
    stream_lds_kernel<false><<<workgroups, kThreads, 0, stream>>>(static_cast<const char*>(src), nchunks,
                                                                  mode == 0 ? 1 : 0, sink);
  return hipGetLastError() == hipSuccess ? TREEPO_OK : TREEPO_EHIP;
}

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
