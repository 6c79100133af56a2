/*
 * sq_probe.h -- C ABI of libsq_probe.so, the roofline probes the benchmark runs beside the
 * rotated W4A4 path to measure what one MI355X sustains on this machine: the int8 matrix-core
 * rate (the peak the W4A4 GEMM is compared against) and HBM bandwidth (the peak of the
 * rotation, quantization and weight-streaming kernels).  Not part of the method.
 *
 * Conventions: device pointers, allocated and owned by the caller; work is enqueued on
 * `stream` (hipStream_t, NULL = default stream) and the caller times and synchronises it.
 * Return value 0 = enqueued, 1 = bad argument, 6 = HIP error (message from
 * sq_probe_last_error()).
 */
#ifndef SQ_PROBE_H_
#define SQ_PROBE_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Message for the last failing call on the calling thread ("" if none). */
const char* sq_probe_last_error(void);

/*
 * sq_probe_mfma_i8 -- back-to-back v_mfma_i32_32x32x32_i8 on registers only, with operand
 * bytes drawn like the W4A4 GEMM's expanded codes (activations 0..15, weights 16 x -7..7),
 * eight independent accumulators per wave, waves_per_simd waves on each SIMD of
 * `workgroups` workgroups of 4 * waves_per_simd waves.
 *   iters          > 0: loop trips; each wave issues 8 * iters MFMAs of 2*32*32*32 int8 ops
 *   workgroups     > 0 (e.g. 256: one per CU)
 *   waves_per_simd 1 or 2
 *   sink           device int32 [workgroups * 4 * waves_per_simd * 64]: a sum of the
 *                  accumulators per lane, so that no MFMA is dead code
 * Ops enqueued: 65536 * 8 * iters * workgroups * 4 * waves_per_simd.
 */
int32_t sq_probe_mfma_i8(int64_t iters, int32_t workgroups, int32_t waves_per_simd, int32_t* sink, void* stream);

/*
 * sq_probe_copy -- dst[i] = src[i] for `bytes` bytes with 16-byte loads and stores, each
 * thread four chunks apart per trip over a grid of `workgroups` x 256 threads.
 *   src, dst   device, 16-byte aligned, not overlapping; bytes > 0, bytes % 16 == 0
 * HBM traffic: bytes read + bytes written.
 */
int32_t sq_probe_copy(const void* src, void* dst, int64_t bytes, int32_t workgroups, void* stream);

/*
 * sq_probe_read -- reads `bytes` bytes with 16-byte loads and writes one xor of them per
 * thread to sink (device uint32 [workgroups * 256]).  src 16-byte aligned, bytes % 16 == 0.
 * HBM traffic: bytes read (+ the sink).
 */
int32_t sq_probe_read(const void* src, int64_t bytes, int32_t workgroups, uint32_t* sink, void* stream);

/*
 * sq_probe_copy_blocks, sq_probe_read_blocks -- the copy and read above, but workgroup b
 * owns one contiguous block of ceil(bytes / 16 / workgroups) 16-byte items and walks it
 * 4 KB at a time (8 copies or 16 reads in flight per thread): each workgroup streams its
 * own region, the access pattern HBM serves fastest.  Arguments, checks and traffic as
 * sq_probe_copy and sq_probe_read.
 */
int32_t sq_probe_copy_blocks(const void* src, void* dst, int64_t bytes, int32_t workgroups, void* stream);
int32_t sq_probe_read_blocks(const void* src, int64_t bytes, int32_t workgroups, uint32_t* sink, void* stream);

/*
 * sq_probe_sleep -- one wave that sleeps (s_sleep) until `microseconds` have passed on the
 * GPU's constant-rate wall clock (hipDeviceAttributeWallClockRate of the current device),
 * and in any case after at most as many sleep steps as wall-clock ticks.  Holds the stream,
 * drawing little power, while the host queues launches that are then to run back to back.
 * microseconds > 0.
 */
int32_t sq_probe_sleep(int64_t microseconds, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SQ_PROBE_H_ */
