/*
 * treepo_bench.h -- measurement probes shipped with the library.
 *
 * These are not part of the decode path.  They give the bandwidth figures
 * that the decode kernels are judged against: a plain device copy of known
 * size (to calibrate hardware byte counters) and a streaming read (the
 * attainable HBM read bandwidth on this device).
 */
#ifndef TREEPO_BENCH_H
#define TREEPO_BENCH_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* dst[0:bytes) = src[0:bytes) on stream.  bytes must be a multiple of 16 and
 * both pointers 16-byte aligned (device memory).  Returns 0 or TREEPO_EINVAL /
 * TREEPO_EHIP. */
int32_t treepo_bench_copy(void* dst, const void* src, size_t bytes, hipStream_t stream);

/* Reads src[0:bytes) once with 16-byte loads and writes one fp32 per
 * workgroup into sink (device, >= 4096 floats) so the reads cannot be elided.
 * Same alignment rules as treepo_bench_copy. */
int32_t treepo_bench_read(const void* src, size_t bytes, float* sink, hipStream_t stream);

/* Streams src[0:bytes) with `workgroups` workgroups of 256 threads and the
 * staging pattern of the decode kernels, writing one fp32 per workgroup into
 * sink (device, >= workgroups floats):
 *   mode 0: each workgroup reads one contiguous share in 16 KiB chunks through
 *           16-byte global->LDS loads, three chunks in flight, a workgroup
 *           barrier per chunk (the decode pipeline);
 *   mode 1: the same staging with chunks assigned grid-stride;
 *   mode 2: each workgroup reads one contiguous share with 16-byte register
 *           loads;
 *   mode 3: mode 0 with the non-temporal hint on every load (exactly the
 *           decode kernels' tile loads).
 * bytes must be a multiple of 16 KiB * workgroups, 1 <= workgroups <= 4096,
 * src 16-byte aligned.  Returns 0, TREEPO_EINVAL or TREEPO_EHIP. */
int32_t treepo_bench_stream(const void* src, size_t bytes, float* sink, int32_t mode,
                            int32_t workgroups, hipStream_t stream);

/* How matrix-core and vector-ALU work share a SIMD.  One workgroup of
 * 256 * waves_per_simd threads (1 <= waves_per_simd <= 4: waves per SIMD);
 * each wave runs `iters` rounds of eight independent
 * v_mfma_f32_16x16x32_bf16 (mode 0), 24 independent fp32 FMAs (mode 1), or
 * both interleaved one MFMA then three FMAs (mode 2), and writes its
 * s_memtime clock delta to cycles[wave] (device, >= 16 uint64) and one float
 * per thread to sink (device, >= 1024 floats).  If the two units overlapped,
 * mode 2 would take about as long as the slower of modes 0 and 1.  Returns
 * 0, TREEPO_EINVAL or TREEPO_EHIP. */
int32_t treepo_bench_overlap(int32_t mode, int32_t waves_per_simd, int32_t iters, float* sink, uint64_t* cycles,
                             hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* TREEPO_BENCH_H */
