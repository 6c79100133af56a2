// Device helpers shared by the HIP kernels: the eq. 1 quantizer's exact fp32 op
// sequence, wave/workgroup reductions, fp16 conversions.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>

namespace sq {

constexpr int kWave = 64;

__device__ __forceinline__ float h2f(uint16_t bits) {
  return __half2float(__ushort_as_half(bits));
}
__device__ __forceinline__ uint16_t f2h(float v) {
  return __half_as_ushort(__float2half_rn(v));
}
// fp16 bits of v rounded to nearest even, saturating at +-65504 (the largest finite fp16)
__device__ __forceinline__ uint16_t f2h_sat(float v) {
  return f2h(fminf(fmaxf(v, -65504.0f), 65504.0f));
}

// Smallest normal fp32 (2^-126).  A group whose alpha would fall below it (zero or
// subnormal: a constant group, or a range under L * 2^-126) is quantized as constant with
// alpha = 1, so 1 / alpha stays finite and every code is 0.
constexpr float kMinNormal = 1.17549435e-38f;

// Asymmetric eq. 1 parameters from a group's min and max, L = 2^bits - 1 levels (15 or 255).
//   r = mx - mn;  alpha = r / L (1 if below kMinNormal);  inv = 1 / alpha  -- each one IEEE rounding.
struct AsymParams {
  float mn, alpha, inv, levels;
};
__device__ __forceinline__ AsymParams asym_params(float mn, float mx, float levels = 15.0f) {
  const float r = __fsub_rn(mx, mn);
  const float a = __fdiv_rn(r, levels);
  const float alpha = (a < kMinNormal) ? 1.0f : a;  // zero or subnormal: constant group
  return {mn, alpha, __fdiv_rn(1.0f, alpha), levels};
}
// t = (v - mn) * inv clamped to [0, L]: rint(t) is then the code
__device__ __forceinline__ float asym_t(float v, const AsymParams& p) {
  return __builtin_amdgcn_fmed3f(__fmul_rn(__fsub_rn(v, p.mn), p.inv), 0.0f, p.levels);
}
// code = clamp(rint((v - mn) * inv), 0, L)
__device__ __forceinline__ uint32_t asym_code(float v, const AsymParams& p) {
  const float t = __fmul_rn(__fsub_rn(v, p.mn), p.inv);
  return static_cast<uint32_t>(fminf(fmaxf(rintf(t), 0.0f), p.levels));
}

// Symmetric eq. 1 (beta = 0, L = 7): alpha = amax / 7 (1 if below kMinNormal); code in [-7, 7].
__device__ __forceinline__ float sym_alpha(float amax) {
  const float a = __fdiv_rn(amax, 7.0f);
  return (a < kMinNormal) ? 1.0f : a;
}
__device__ __forceinline__ int sym_code(float v, float inv) {
  return static_cast<int>(fminf(fmaxf(rintf(__fmul_rn(v, inv)), -7.0f), 7.0f));
}

__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fminf(v, __shfl_xor(v, m, kWave));
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, kWave));
  return v;
}
__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

}  // namespace sq
