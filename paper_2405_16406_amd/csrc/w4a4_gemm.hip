// int4 x int4 GEMM on the int8 matrix cores of gfx950 with the dequantising epilogue.
//
// acc[m,n] = sum_k qa[m,k] qw[n,k] (exact, int32), y = fp16(s_n (alpha_m acc + beta_m rs_n) + bias_n).
//
// Codes arrive packed two per byte (even k in the low nibble).  Both operands are
// expanded to int8 in registers just before v_mfma_i32_32x32x32_i8:
//   activations (0..15):  lo = d & 0x0F0F0F0F,         hi = (d >> 4) & 0x0F0F0F0F
//   weights (-7..7):      lo = (d << 4) & 0xF0F0F0F0,  hi = d & 0xF0F0F0F0     (= 16 * code)
// so each int8 byte holds one code (weights scaled by 16, which is exact) and the
// accumulator is 16 * acc; an arithmetic shift by 4 recovers acc exactly.  A and B are
// expanded with the same byte order, so the k permutation this introduces cancels in
// the dot product.
//
// Tiling: 256 threads (4 waves) per 128x128 output tile, 64-k slices staged in LDS
// (packed, row pitch 40 bytes so a 16-lane group of 8-byte fragment reads touches 16
// distinct bank pairs), each wave owns a 64x64 sub-tile = 2x2 MFMA blocks of 32x32.
#include "sq_device.h"
#include "sq_internal.h"

namespace sq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kBM = 128;
constexpr int kBN = 128;
constexpr int kBKB = 32;     // packed bytes per row per k slice (64 k)
constexpr int kPitch = 40;   // LDS row pitch in bytes
constexpr int kThreads = 256;

__device__ __forceinline__ v4i expand_act(uint2 d) {
  v4i r;
  r[0] = static_cast<int>(d.x & 0x0F0F0F0Fu);
  r[1] = static_cast<int>((d.x >> 4) & 0x0F0F0F0Fu);
  r[2] = static_cast<int>(d.y & 0x0F0F0F0Fu);
  r[3] = static_cast<int>((d.y >> 4) & 0x0F0F0F0Fu);
  return r;
}
__device__ __forceinline__ v4i expand_wgt(uint2 d) {
  v4i r;
  r[0] = static_cast<int>((d.x << 4) & 0xF0F0F0F0u);
  r[1] = static_cast<int>(d.x & 0xF0F0F0F0u);
  r[2] = static_cast<int>((d.y << 4) & 0xF0F0F0F0u);
  r[3] = static_cast<int>(d.y & 0xF0F0F0F0u);
  return r;
}

__global__ void __launch_bounds__(kThreads)
w4a4_gemm_v1(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) uint8_t As[kBM * kPitch];
  __shared__ __attribute__((aligned(16))) uint8_t Bs[kBN * kPitch];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * kBM;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * kBN;
  const int wm = (wave >> 1) * 64;
  const int wn = (wave & 1) * 64;
  const int64_t KB = g.K / 2;

  v16i acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0;

  const int lr = tid >> 1;          // tile row this thread stages
  const int lc = (tid & 1) * 16;    // byte offset within the 32-byte slice
  const int64_t am = m0 + lr;
  const int64_t bn = n0 + lr;
  const uint8_t* arow = g.xq + am * KB + lc;
  const uint8_t* brow = g.wq + bn * KB + lc;
  const bool aok = am < g.M;
  const bool bok = bn < g.N;

  for (int64_t kb = 0; kb < KB; kb += kBKB) {
    uint4 va = make_uint4(0, 0, 0, 0);
    uint4 vb = make_uint4(0, 0, 0, 0);
    if (aok) va = *reinterpret_cast<const uint4*>(arow + kb);
    if (bok) vb = *reinterpret_cast<const uint4*>(brow + kb);
    __syncthreads();
    *reinterpret_cast<uint2*>(As + lr * kPitch + lc) = make_uint2(va.x, va.y);
    *reinterpret_cast<uint2*>(As + lr * kPitch + lc + 8) = make_uint2(va.z, va.w);
    *reinterpret_cast<uint2*>(Bs + lr * kPitch + lc) = make_uint2(vb.x, vb.y);
    *reinterpret_cast<uint2*>(Bs + lr * kPitch + lc + 8) = make_uint2(vb.z, vb.w);
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int off = ks * 16 + (lane >> 5) * 8;
      v4i af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int r = wm + i * 32 + (lane & 31);
        af[i] = expand_act(*reinterpret_cast<const uint2*>(As + r * kPitch + off));
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int r = wn + j * 32 + (lane & 31);
        bf[j] = expand_wgt(*reinterpret_cast<const uint2*>(Bs + r * kPitch + off));
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
  }

  // epilogue: lane holds C[8*(r/4) + 4*(lane/32) + r%4][lane%32] of each 32x32 block
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int64_t n = n0 + wn + j * 32 + (lane & 31);
    if (n >= g.N) continue;
    const float sn = g.wa[n];
    const float rsn = static_cast<float>(g.rs[n]);
    const float bn_ = g.bias ? h2f(g.bias[n]) : 0.0f;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + wm + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m >= g.M) continue;
        const int a = acc[i][j][r] >> 4;
        if (g.dbg_acc) g.dbg_acc[m * g.N + n] = a;
        const float t = __fadd_rn(__fmul_rn(g.xa[m], static_cast<float>(a)), __fmul_rn(g.xb[m], rsn));
        float yv = __fmul_rn(sn, t);
        if (g.bias) yv = __fadd_rn(yv, bn_);
        g.y[m * g.ldy + n] = f2h(yv);
      }
    }
  }
}

}  // namespace

hipError_t launch_w4a4_gemm(const GemmArgs& g, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>((g.N + kBN - 1) / kBN), static_cast<unsigned>((g.M + kBM - 1) / kBM));
  hipLaunchKernelGGL(w4a4_gemm_v1, grid, dim3(kThreads), 0, stream, g);
  return hipGetLastError();
}

}  // namespace sq
