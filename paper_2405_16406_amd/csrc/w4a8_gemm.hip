// W4A8 linear layer: 8-bit asymmetric per-token activation codes (eq. 1, L = 255) against the
// packed 4-bit per-channel weights, the W4A8 setting of the main results and of the speed
// measurement (Sec. 4.2, 4.5).  acc[m,n] = sum_k qa[m,k] qw[n,k] exactly, and the epilogue
// expands eq. 1 on both operands as the W4A4 one does:
//     y = fp16( s_n (alpha_m acc + beta_m rs_n) + bias_n ).
// The int8 MFMA takes signed bytes, so the codes enter as qa - 128 and the shift moves into
// the zero-point term: alpha_m acc + beta_m rs_n = alpha_m acc' + (beta_m + 128 alpha_m) rs_n.
//
// 128 x 128 tiles, 4 waves of 64 x 64 (2 x 2 blocks of 32 x 32), 64 k per stage: A rows of 64
// code bytes and B rows of 32 packed bytes pass through LDS (two buffers; the next stage is
// loaded into registers while this one is multiplied).  The weights are the MFMA A operand,
// expanded to 16 x code as in the W4A4 kernels (k-slot order k0 k2 k4 k6 | k1 k3 k5 k7 |
// k8 ...); v_perm_b32 puts the activation bytes in the same order and an xor with 0x80 makes
// them signed.  A lane then holds output row m and four consecutive columns per register quad.
#include "sq_device.h"
#include "sq_internal.h"

namespace sq {
namespace {

constexpr int kBM = 128, kBN = 128, kBK = 64;  // tile rows (tokens), columns (outputs), k per stage
constexpr int kAPitch = kBK + 16;              // LDS bytes per activation row (padded)
constexpr int kBPitch = kBK / 2 + 8;           // LDS bytes per packed weight row (padded)
constexpr int kAStage = kBM * kAPitch, kBStage = kBN * kBPitch;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

// 16 activation codes k0..k15 (natural order) -> signed MFMA operand in the weights' order
__device__ __forceinline__ v4i act_operand(const v4u d) {
  const uint32_t f = 0x80808080u;
  return v4i{static_cast<int>(__builtin_amdgcn_perm(d[1], d[0], 0x06040200u) ^ f),
             static_cast<int>(__builtin_amdgcn_perm(d[1], d[0], 0x07050301u) ^ f),
             static_cast<int>(__builtin_amdgcn_perm(d[3], d[2], 0x06040200u) ^ f),
             static_cast<int>(__builtin_amdgcn_perm(d[3], d[2], 0x07050301u) ^ f)};
}

// 16 packed weight codes (8 bytes, even k in the low nibble) -> 16 x code, same order
__device__ __forceinline__ v4i wgt_operand(const uint2 d) {
  return v4i{static_cast<int>((d.x << 4) & 0xF0F0F0F0u), static_cast<int>(d.x & 0xF0F0F0F0u),
             static_cast<int>((d.y << 4) & 0xF0F0F0F0u), static_cast<int>(d.y & 0xF0F0F0F0u)};
}

__global__ void __launch_bounds__(256)
w4a8_gemm_tile(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * (kAStage + kBStage)];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c = lane & 31, h = lane >> 5;
  const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * kBM;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * kBN;
  const int64_t K = g.K, KB = g.K / 2;
  const int nst = static_cast<int>(K / kBK);

  // stage loads: activation chunk j of this thread = 16 bytes (row (tid + 256 j) / 4,
  // column 16 ((tid + 256 j) % 4)); weight chunk = 16 bytes (row tid / 2, half tid % 2)
  v4u ra[2], rb;
  auto gload = [&](int st) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int ch = tid + 256 * j;
      const int64_t m = m0 + ch / 4;
      ra[j] = m < g.M ? *reinterpret_cast<const v4u*>(g.xq + m * K + st * kBK + 16 * (ch % 4)) : v4u{0u, 0u, 0u, 0u};
    }
    const int64_t n = n0 + tid / 2;
    rb = n < g.N ? *reinterpret_cast<const v4u*>(g.wq + n * KB + st * (kBK / 2) + 16 * (tid % 2)) : v4u{0u, 0u, 0u, 0u};
  };
  auto lstore = [&](int buf) {
    uint8_t* As = lds + buf * (kAStage + kBStage);
    uint8_t* Bs = As + kAStage;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int ch = tid + 256 * j;
      *reinterpret_cast<v4u*>(As + (ch / 4) * kAPitch + 16 * (ch % 4)) = ra[j];
    }
    *reinterpret_cast<v4u*>(Bs + (tid / 2) * kBPitch + 16 * (tid % 2)) = rb;
  };

  v16i acc[2][2];  // [weight block j][activation block i]
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][i][r] = 0;

  gload(0);
  lstore(0);
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const bool more = st + 1 < nst;
    if (more) gload(st + 1);
    const uint8_t* As = lds + (st & 1) * (kAStage + kBStage);
    const uint8_t* Bs = As + kAStage;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {  // two MFMA k-steps of 32
      v4i af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = act_operand(*reinterpret_cast<const v4u*>(As + (wm + 32 * i + c) * kAPitch + 32 * ks + 16 * h));
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bf[j] = wgt_operand(*reinterpret_cast<const uint2*>(Bs + (wn + 32 * j + c) * kBPitch + 16 * ks + 8 * h));
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < 2; ++i) acc[j][i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(bf[j], af[i], acc[j][i], 0, 0, 0);
    }
    if (more) lstore((st + 1) & 1);
    __syncthreads();
  }

  // epilogue: lane (c, h), register r of block (j, i) holds acc' = 16 sum (qa - 128) qw for
  // row m = wm + 32 i + c, column n = wn + 32 j + 8 (r / 4) + 4 h + r % 4
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int64_t m = m0 + wm + 32 * i + c;
    if (m >= g.M) continue;
    const float xa = g.xa[m];
    const float ra16 = __fmul_rn(xa, 0.0625f);
    const float rb = __fmaf_rn(128.0f, xa, g.xb[m]);  // beta + 128 alpha
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t n = n0 + wn + 32 * j + 8 * (r >> 2) + 4 * h + (r & 3);
        if (n >= g.N) continue;
        const float s = g.wa[n];
        const float t = __fmul_rn(s, static_cast<float>(acc[j][i][r]));
        const float bias = g.bias ? h2f(g.bias[n]) : 0.0f;
        const float yv = __fmaf_rn(ra16, t, __fmaf_rn(rb, __fmul_rn(s, static_cast<float>(g.rs[n])), bias));
        g.y[m * g.ldy + n] = f2h(yv);
        if (g.dbg_acc) g.dbg_acc[m * g.N + n] = (acc[j][i][r] >> 4) + 128 * g.rs[n];
      }
  }
}

}  // namespace

hipError_t launch_w4a8_gemm(const GemmArgs& g, hipStream_t stream) {
  // decode-sized M: the weight-streaming kernel with 8-bit activations
  const hipError_t e = launch_w4a8_skinny(g, stream);
  if (e != hipErrorNotSupported) return e;
  const dim3 grid(static_cast<unsigned>((g.N + kBN - 1) / kBN), static_cast<unsigned>((g.M + kBM - 1) / kBM));
  return launch(w4a8_gemm_tile, grid, dim3(256), 0, stream, g);
}

}  // namespace sq
