// W4A8 linear layer: 8-bit asymmetric per-token activation codes (eq. 1, L = 255) against the
// packed 4-bit per-channel weights, the W4A8 setting of the main results and of the speed
// measurement (Sec. 4.2, 4.5).  acc[m,n] = sum_k qa[m,k] qw[n,k] exactly, and the epilogue
// expands eq. 1 on both operands as the W4A4 one does:
//     y = fp16( s_n (alpha_m acc + beta_m rs_n) + bias_n ).
// The int8 MFMA takes signed bytes, so the codes enter as qa - 128 and the shift moves into
// the zero-point term: alpha_m acc + beta_m rs_n = alpha_m acc' + (beta_m + 128 alpha_m) rs_n.
//
// 128 x BN tiles (BN = 128 or 256), 4 waves of 64 x BN/2 (blocks of 32 x 32), BK = 64 or 128
// k per stage: activation rows of BK code bytes and weight rows of BK/2 packed bytes pass
// through LDS (two buffers; the next stage is loaded into registers while this one is
// multiplied).  The weights are the MFMA A operand, expanded to 16 x code as in the W4A4
// kernels (k-slot order k0 k2 k4 k6 | k1 k3 k5 k7 | k8 ...); v_perm_b32 puts the activation
// bytes in the same order and an xor with 0x80 makes them signed, once per chunk as it is
// stored to LDS.  A lane then holds output row m and four consecutive columns per register
// quad.
#include "sq_device.h"
#include "sq_internal.h"


namespace sq {
namespace {

constexpr int kBM = 128;  // tile rows (tokens)

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

// LDS geometry of a BN x BK stage: activation rows of BK code bytes padded by 16 and weight
// rows of BK/2 packed bytes padded by 8, so that the 32 rows one fragment read touches start
// on distinct bank groups (16-byte reads: row pitch 4 mod 16 dwords; 8-byte reads: 2 mod 4)
template <int BN, int BK>
struct Tile {
  static constexpr int APitch = BK + 16;
  static constexpr int BPitch = BK / 2 + 8;
  static constexpr int AStage = kBM * APitch;
  static constexpr int BStage = BN * BPitch;
  static constexpr int LDS = 2 * (AStage + BStage);
  static constexpr int ACH = kBM * BK / 16 / 256;      // 16-byte activation chunks per thread
  static constexpr int BCH = BN * BK / 32 / 256;       // 16-byte weight chunks per thread
  static constexpr int AROW = BK / 16, BROW = BK / 32;  // chunks per row
  static constexpr int NB = BN / 64;                    // 32-wide weight blocks per wave
  static_assert(ACH >= 1 && BCH >= 1 && BK % 32 == 0, "tile");
};

// 16 activation codes k0..k15 (natural order) -> signed MFMA operand in the weights' order;
// applied once per chunk as it goes to LDS, so the waves that read it take it as is
__device__ __forceinline__ v4u act_operand(const v4u d) {
  const uint32_t f = 0x80808080u;
  return v4u{__builtin_amdgcn_perm(d[1], d[0], 0x06040200u) ^ f, __builtin_amdgcn_perm(d[1], d[0], 0x07050301u) ^ f,
             __builtin_amdgcn_perm(d[3], d[2], 0x06040200u) ^ f, __builtin_amdgcn_perm(d[3], d[2], 0x07050301u) ^ f};
}

// 16 packed weight codes (8 bytes, even k in the low nibble) -> 16 x code, same order
__device__ __forceinline__ v4i wgt_operand(const uint2 d) {
  return v4i{static_cast<int>((d.x << 4) & 0xF0F0F0F0u), static_cast<int>(d.x & 0xF0F0F0F0u),
             static_cast<int>((d.y << 4) & 0xF0F0F0F0u), static_cast<int>(d.y & 0xF0F0F0F0u)};
}

template <int BN, int BK>
__global__ void __launch_bounds__(256, BN == 256 ? 2 : 1)  // wide tiles: two workgroups per CU
w4a8_gemm_tile(GemmArgs g) {
  using T = Tile<BN, BK>;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c = lane & 31, h = lane >> 5;
  const int wm = (wave >> 1) * 64, wn = (wave & 1) * (BN / 2);
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * kBM;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * BN;
  const int64_t K = g.K, KB = g.K / 2;
  const int nst = static_cast<int>(K / BK);

  // stage loads: activation chunk ch = tid + 256 j is row ch / AROW, 16 bytes at
  // 16 (ch % AROW); weight chunk ch is row ch / BROW, 16 bytes at 16 (ch % BROW)
  v4u ra[T::ACH], rb[T::BCH];
  auto gload = [&](int st) {
#pragma unroll
    for (int j = 0; j < T::ACH; ++j) {
      const int ch = tid + 256 * j;
      const int64_t m = m0 + ch / T::AROW;
      ra[j] = m < g.M ? *reinterpret_cast<const v4u*>(g.xq + m * K + st * BK + 16 * (ch % T::AROW))
                      : v4u{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < T::BCH; ++j) {
      const int ch = tid + 256 * j;
      const int64_t n = n0 + ch / T::BROW;
      rb[j] = n < g.N ? *reinterpret_cast<const v4u*>(g.wq + n * KB + st * (BK / 2) + 16 * (ch % T::BROW))
                      : v4u{0u, 0u, 0u, 0u};
    }
  };
  auto lstore = [&](int buf) {
    uint8_t* As = lds + buf * (T::AStage + T::BStage);
    uint8_t* Bs = As + T::AStage;
#pragma unroll
    for (int j = 0; j < T::ACH; ++j) {
      const int ch = tid + 256 * j;
      *reinterpret_cast<v4u*>(As + (ch / T::AROW) * T::APitch + 16 * (ch % T::AROW)) = act_operand(ra[j]);
    }
#pragma unroll
    for (int j = 0; j < T::BCH; ++j) {
      const int ch = tid + 256 * j;
      *reinterpret_cast<v4u*>(Bs + (ch / T::BROW) * T::BPitch + 16 * (ch % T::BROW)) = rb[j];
    }
  };

  v16i acc[T::NB][2];  // [weight block j][activation block i]
#pragma unroll
  for (int j = 0; j < T::NB; ++j)
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
    const uint8_t* As = lds + (st & 1) * (T::AStage + T::BStage);
    const uint8_t* Bs = As + T::AStage;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {  // MFMA k-steps of 32
      v4i af[2], bf[T::NB];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const v4i*>(As + (wm + 32 * i + c) * T::APitch + 32 * ks + 16 * h);
#pragma unroll
      for (int j = 0; j < T::NB; ++j)
        bf[j] = wgt_operand(*reinterpret_cast<const uint2*>(Bs + (wn + 32 * j + c) * T::BPitch + 16 * ks + 8 * h));
#pragma unroll
      for (int j = 0; j < T::NB; ++j)
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
    const float rbeta = __fmaf_rn(128.0f, xa, g.xb[m]);  // beta + 128 alpha
#pragma unroll
    for (int j = 0; j < T::NB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t n = n0 + wn + 32 * j + 8 * (r >> 2) + 4 * h + (r & 3);
        if (n >= g.N) continue;
        const float s = g.wa[n];
        const float t = __fmul_rn(s, static_cast<float>(acc[j][i][r]));
        const float bias = g.bias ? h2f(g.bias[n]) : 0.0f;
        const float yv = __fmaf_rn(ra16, t, __fmaf_rn(rbeta, __fmul_rn(s, static_cast<float>(g.rs[n])), bias));
        g.y[m * g.ldy + n] = f2h(yv);
        if (g.dbg_acc) g.dbg_acc[m * g.N + n] = (acc[j][i][r] >> 4) + 128 * g.rs[n];
      }
  }
}

template <int BN, int BK>
hipError_t launch_tile(const GemmArgs& g, hipStream_t stream) {
  using T = Tile<BN, BK>;
  constexpr auto kern = w4a8_gemm_tile<BN, BK>;
  const hipError_t init = set_max_lds<kern>(T::LDS);
  if (init != hipSuccess) return init;
  const dim3 grid(static_cast<unsigned>((g.N + BN - 1) / BN), static_cast<unsigned>((g.M + kBM - 1) / kBM));
  return launch(kern, grid, dim3(256), T::LDS, stream, g);
}

}  // namespace

hipError_t launch_w4a8_gemm(const GemmArgs& g, hipStream_t stream) {
  // decode-sized M: the weight-streaming kernel with 8-bit activations
  const hipError_t e = launch_w4a8_skinny(g, stream);
  if (e != hipErrorNotSupported) return e;
  // prefill: the LDS-ring kernel of the W4A4 GEMM with 8-bit A blocks; this file's
  // register-staged tiles where its 32-bit buffer offsets do not cover the operands
  // (operands of 2 GB and more)
  const hipError_t r = launch_w4a8_ring(g, stream);
  if (r != hipErrorNotSupported) return r;
  // Measured on MI355X (us, tiles 128x64 / 128x128 / 256x64 / 256x128 in N x k-stage):
  //   [2048 x 22016 x 4096]  404 / 401 / 417 / 387      [2048 x 4096 x 11008]  181 / 165 / 221 / 186
  //   [4096 x 28672 x 4096]  944 / 916 / 920 / 846      [4096 x 4096 x 14336]  446 / 397 / 390 / 362
  // 128-deep stages need K % 128 == 0; 256-wide tiles pay off from two workgroups per CU.
  if (g.K % 128 != 0) return launch_tile<128, 64>(g, stream);
  const int64_t wide = ((g.M + kBM - 1) / kBM) * ((g.N + 255) / 256);
  if (wide >= 512) return launch_tile<256, 128>(g, stream);
  return launch_tile<128, 128>(g, stream);
}

}  // namespace sq
