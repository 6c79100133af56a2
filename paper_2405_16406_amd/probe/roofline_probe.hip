// Roofline probes (include/sq_probe.h): an int8 matrix-core loop and HBM copy / read
// streams, measured on the box beside the datasheet peaks.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "sq_probe.h"

namespace {

thread_local std::string g_err;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

// small deterministic hash of (lane, index): operand bytes that change per lane and set
__device__ __forceinline__ uint32_t mix(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

// 4 activation operand sets (bytes 0..15) and 2 weight sets (bytes 16 x -7..7), eight
// accumulators: each trip issues the 8 products a[i % 4] x b[i / 4]
__global__ void __launch_bounds__(512) probe_mfma_i8(int64_t iters, int32_t* sink) {
  const uint32_t lane = threadIdx.x;
  v4i a[4], b[2];
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int r = 0; r < 4; ++r) a[s][r] = static_cast<int>(mix(lane * 97u + s * 13u + r) & 0x0F0F0F0Fu);
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      uint32_t w = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = static_cast<int>(mix(lane * 131u + s * 17u + r * 4u + e) % 15u) - 7;  // -7..7
        w |= (static_cast<uint32_t>(c * 16) & 0xFFu) << (8 * e);
      }
      b[s][r] = static_cast<int>(w);
    }
  v16i acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0;
  for (int64_t t = 0; t < iters; ++t) {
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i & 3], b[i >> 2], acc[i], 0, 0, 0);
  }
  int s = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[i][r];
  sink[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ void __launch_bounds__(256) probe_copy(const v4u* __restrict__ src, v4u* __restrict__ dst, int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const v4u x0 = src[i], x1 = src[i + stride], x2 = src[i + 2 * stride], x3 = src[i + 3 * stride];
    dst[i] = x0;
    dst[i + stride] = x1;
    dst[i + 2 * stride] = x2;
    dst[i + 3 * stride] = x3;
  }
  for (; i < n; i += stride) dst[i] = src[i];
}

__global__ void __launch_bounds__(256) probe_read(const v4u* __restrict__ src, int64_t n, uint32_t* sink) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  v4u acc = {0u, 0u, 0u, 0u};
  for (; i + 3 * stride < n; i += 4 * stride) {
    const v4u x0 = src[i], x1 = src[i + stride], x2 = src[i + 2 * stride], x3 = src[i + 3 * stride];
    acc ^= x0 ^ x1 ^ x2 ^ x3;
  }
  for (; i < n; i += stride) acc ^= src[i];
  sink[blockIdx.x * blockDim.x + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

// Streams: workgroup b owns the contiguous items [b * per, min((b + 1) * per, n)) and walks
// them 256 items (4 KB) at a time, 16 loads in flight per thread.
__global__ void __launch_bounds__(256) probe_read_blocks(const v4u* __restrict__ src, int64_t n, int64_t per,
                                                         uint32_t* sink) {
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * per;
  const int64_t b1 = b0 + per < n ? b0 + per : n;
  v4u acc = {0u, 0u, 0u, 0u};
  int64_t i = b0 + threadIdx.x;
  for (; i + 15 * 256 < b1; i += 16 * 256) {
    v4u x[16];
#pragma unroll
    for (int d = 0; d < 16; ++d) x[d] = src[i + d * 256];
#pragma unroll
    for (int d = 0; d < 16; ++d) acc ^= x[d];
  }
  for (; i < b1; i += 256) acc ^= src[i];
  sink[blockIdx.x * blockDim.x + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}
__global__ void __launch_bounds__(256) probe_copy_blocks(const v4u* __restrict__ src, v4u* __restrict__ dst,
                                                         int64_t n, int64_t per) {
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * per;
  const int64_t b1 = b0 + per < n ? b0 + per : n;
  int64_t i = b0 + threadIdx.x;
  for (; i + 7 * 256 < b1; i += 8 * 256) {
    v4u x[8];
#pragma unroll
    for (int d = 0; d < 8; ++d) x[d] = src[i + d * 256];
#pragma unroll
    for (int d = 0; d < 8; ++d) dst[i + d * 256] = x[d];
  }
  for (; i < b1; i += 256) dst[i] = src[i];
}
// bounded wait: ends when the wall clock has advanced `ticks` or after `ticks` sleeps of
// about 64 cycles each, whichever comes first
__global__ void __launch_bounds__(64) probe_sleep(int64_t ticks) {
  const uint64_t t0 = wall_clock64();
  for (int64_t i = 0; i < ticks; ++i) {
    if (wall_clock64() - t0 >= static_cast<uint64_t>(ticks)) break;
    __builtin_amdgcn_s_sleep(1);
  }
}

int32_t hip_result(hipError_t e, const char* what) {
  if (e == hipSuccess) {
    g_err.clear();
    return 0;
  }
  g_err = std::string(what) + ": " + hipGetErrorString(e);
  return 6;
}

int32_t bad(const char* msg) {
  g_err = msg;
  return 1;
}

}  // namespace

extern "C" {

const char* sq_probe_last_error(void) { return g_err.c_str(); }

int32_t sq_probe_mfma_i8(int64_t iters, int32_t workgroups, int32_t waves_per_simd, int32_t* sink, void* stream) {
  if (iters <= 0 || workgroups <= 0 || (waves_per_simd != 1 && waves_per_simd != 2) || !sink)
    return bad("iters > 0, workgroups > 0, waves_per_simd 1 or 2 and a sink are required");
  hipLaunchKernelGGL(probe_mfma_i8, dim3(workgroups), dim3(256 * waves_per_simd), 0,
                     static_cast<hipStream_t>(stream), iters, sink);
  return hip_result(hipGetLastError(), "probe_mfma_i8 launch");
}

int32_t sq_probe_copy(const void* src, void* dst, int64_t bytes, int32_t workgroups, void* stream) {
  if (!src || !dst || bytes <= 0 || bytes % 16 || workgroups <= 0 ||
      (reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 16)
    return bad("16-byte aligned src and dst, bytes > 0 and a multiple of 16, workgroups > 0");
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (s0 < d0 + static_cast<uint64_t>(bytes) && d0 < s0 + static_cast<uint64_t>(bytes)) return bad("src and dst overlap");
  hipLaunchKernelGGL(probe_copy, dim3(workgroups), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const v4u*>(src), static_cast<v4u*>(dst), bytes / 16);
  return hip_result(hipGetLastError(), "probe_copy launch");
}

int32_t sq_probe_read(const void* src, int64_t bytes, int32_t workgroups, uint32_t* sink, void* stream) {
  if (!src || !sink || bytes <= 0 || bytes % 16 || workgroups <= 0 || reinterpret_cast<uintptr_t>(src) % 16)
    return bad("16-byte aligned src, bytes > 0 and a multiple of 16, workgroups > 0, a sink");
  hipLaunchKernelGGL(probe_read, dim3(workgroups), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const v4u*>(src), bytes / 16, sink);
  return hip_result(hipGetLastError(), "probe_read launch");
}

int32_t sq_probe_read_blocks(const void* src, int64_t bytes, int32_t workgroups, uint32_t* sink, void* stream) {
  if (!src || !sink || bytes <= 0 || bytes % 16 || workgroups <= 0 || reinterpret_cast<uintptr_t>(src) % 16)
    return bad("16-byte aligned src, bytes > 0 and a multiple of 16, workgroups > 0, a sink");
  const int64_t n = bytes / 16, per = (n + workgroups - 1) / workgroups;
  hipLaunchKernelGGL(probe_read_blocks, dim3(workgroups), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const v4u*>(src), n, per, sink);
  return hip_result(hipGetLastError(), "probe_read_blocks launch");
}
int32_t sq_probe_copy_blocks(const void* src, void* dst, int64_t bytes, int32_t workgroups, void* stream) {
  if (!src || !dst || bytes <= 0 || bytes % 16 || workgroups <= 0 ||
      (reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 16)
    return bad("16-byte aligned src and dst, bytes > 0 and a multiple of 16, workgroups > 0");
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (s0 < d0 + static_cast<uint64_t>(bytes) && d0 < s0 + static_cast<uint64_t>(bytes)) return bad("src and dst overlap");
  const int64_t n = bytes / 16, per = (n + workgroups - 1) / workgroups;
  hipLaunchKernelGGL(probe_copy_blocks, dim3(workgroups), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const v4u*>(src), static_cast<v4u*>(dst), n, per);
  return hip_result(hipGetLastError(), "probe_copy_blocks launch");
}
int32_t sq_probe_sleep(int64_t microseconds, void* stream) {
  if (microseconds <= 0) return bad("microseconds > 0");
  int dev = 0, khz = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
  if (e != hipSuccess) return hip_result(e, "wall clock rate");
  if (khz <= 0) return bad("no wall clock rate");
  hipLaunchKernelGGL(probe_sleep, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream),
                     microseconds * khz / 1000);
  return hip_result(hipGetLastError(), "probe_sleep launch");
}

}  // extern "C"
