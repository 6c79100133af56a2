// R3 on post-RoPE Q and K (Sec. 3.1) fused with 4-bit asymmetric K/V cache quantization.
//
// One head vector (D = 128 fp16) is one quantization group.  Sixteen lanes own a
// group, eight contiguous elements each (one 16-byte load per tensor).  The 128-point
// Walsh-Hadamard transform is three in-register butterfly stages (element strides 1, 2,
// 4) followed by four cross-lane stages (lane xor 1, 2, 4, 8); min/max use the same
// 16-lane butterflies.  Each lane writes 8 codes as one 32-bit store.
#include "sq_device.h"
#include "sq_internal.h"

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kLanesPerGroup = 16;
constexpr int kD = 128;

__device__ __forceinline__ void load8(const uint16_t* p, float (&e)[8]) {
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    e[2 * i] = h2f(static_cast<uint16_t>(w[i] & 0xFFFFu));
    e[2 * i + 1] = h2f(static_cast<uint16_t>(w[i] >> 16));
  }
}

__device__ __forceinline__ void fwht128(float (&e)[8], int sl) {
#pragma unroll
  for (int h = 1; h < 8; h <<= 1) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if ((i & h) == 0) {
        const float u = e[i], w = e[i + h];
        e[i] = __fadd_rn(u, w);
        e[i + h] = __fsub_rn(u, w);
      }
    }
  }
#pragma unroll
  for (int m = 1; m < kLanesPerGroup; m <<= 1) {
    const bool upper = (sl & m) != 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float p = __shfl_xor(e[i], m, kLanesPerGroup);
      e[i] = upper ? __fsub_rn(p, e[i]) : __fadd_rn(e[i], p);
    }
  }
}

__device__ __forceinline__ void quant_store(const float (&e)[8], int sl, int64_t grp, uint8_t* q,
                                            float* alpha, float* beta) {
  float mn = e[0], mx = e[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) {
    mn = fminf(mn, e[i]);
    mx = fmaxf(mx, e[i]);
  }
#pragma unroll
  for (int m = 1; m < kLanesPerGroup; m <<= 1) {
    mn = fminf(mn, __shfl_xor(mn, m, kLanesPerGroup));
    mx = fmaxf(mx, __shfl_xor(mx, m, kLanesPerGroup));
  }
  const AsymParams p = asym_params(mn, mx);
  uint32_t word = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) word |= asym_code(e[i], p) << (4 * i);
  *reinterpret_cast<uint32_t*>(q + grp * (kD / 2) + sl * 4) = word;
  if (sl == 0) {
    alpha[grp] = p.alpha;
    beta[grp] = p.mn;
  }
}

__global__ void __launch_bounds__(kThreads)
qk_had_kvquant_v1(KvArgs a) {
  const int64_t grp = (static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x) / kLanesPerGroup;
  const int sl = threadIdx.x & (kLanesPerGroup - 1);
  if (grp >= a.groups) return;  // all 16 lanes of a group leave together
  const int64_t off = grp * kD + sl * 8;
  float e[8];

  load8(a.q + off, e);
  fwht128(e, sl);
  uint32_t packed[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    packed[i] = static_cast<uint32_t>(f2h(__fmul_rn(e[2 * i], a.inv_sqrt_d))) |
                (static_cast<uint32_t>(f2h(__fmul_rn(e[2 * i + 1], a.inv_sqrt_d))) << 16);
  }
  *reinterpret_cast<uint4*>(a.q_rot + off) = make_uint4(packed[0], packed[1], packed[2], packed[3]);

  load8(a.k + off, e);
  fwht128(e, sl);
#pragma unroll
  for (int i = 0; i < 8; ++i) e[i] = __fmul_rn(e[i], a.inv_sqrt_d);
  if (a.dbg_k) {
#pragma unroll
    for (int i = 0; i < 8; ++i) a.dbg_k[off + i] = e[i];
  }
  quant_store(e, sl, grp, a.kq, a.ka, a.kb);

  load8(a.v + off, e);
  quant_store(e, sl, grp, a.vq, a.va, a.vb);
}

}  // namespace

hipError_t launch_qk_had_kvquant(const KvArgs& a, hipStream_t stream) {
  const int64_t threads = a.groups * kLanesPerGroup;
  const unsigned blocks = static_cast<unsigned>((threads + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(qk_had_kvquant_v1, dim3(blocks), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sq
