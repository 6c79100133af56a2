// Online Hadamard rotation of rows fused with 4-bit quantization (eq. 1, Sec. 2).
//
// Generic kernel: one workgroup of 256 threads per row.  The rotated row lives in LDS
// as fp32.  Each contiguous block of n = a*b elements is multiplied by
// (H_a (x) S_b) / sqrt(n) with element i = i_a*b + i_b:
//   1. dense stage  Y[j_a][i_b] = sum_{i_a} x[i_a*b + i_b] H[i_a][j_a]   (fp32, from L1/L2)
//   2. Walsh-Hadamard butterflies over i_b (contiguous), one LDS pass per stage
//   3. scale by fl32(1/sqrt(n))
// then the quantizer: asymmetric per group (activations) or symmetric per row with the
// code row sum (weights).  Variants: a +-1 diagonal S in front of the rotation (the random
// Hadamard matrix S H of Sec. 2.2) flips the sign of input element i when S[i % n] < 0,
// which is exact; a clipping ratio r < 1 quantizes the range [r min, r max] of each group
// (App. A "Quantization choice") with the codes outside it clamped.
#include "sq_device.h"
#include "sq_internal.h"

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

__device__ float block_min(float v, float* red) {
  v = wave_min(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) r = fminf(r, red[i]);
  return r;
}
__device__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) r = fmaxf(r, red[i]);
  return r;
}
__device__ int block_sum(int v, int* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) red[w] = v;
  __syncthreads();
  int r = 0;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) r += red[i];
  return r;
}

// fp16 element i of a row, its sign flipped where S[i % n] < 0 (signs may be null)
__device__ __forceinline__ float signed_elem(const uint16_t* __restrict__ xr, int i,
                                            const int8_t* __restrict__ signs, int n) {
  uint16_t v = xr[i];
  if (signs && signs[i % n] < 0) v ^= 0x8000u;
  return h2f(v);
}

// Fills buf[0..K) with the rotated row (fp32).  Ends with a barrier.
__device__ void rotate_row_to_lds(const uint16_t* __restrict__ xr, int K, int a,
                                  const int8_t* __restrict__ H, int b, float inv_sqrt_n,
                                  const int8_t* __restrict__ signs, float* __restrict__ buf) {
  const int n = a * b;
  if (a == 1) {
    for (int i = threadIdx.x; i < K; i += kThreads) buf[i] = signed_elem(xr, i, signs, n);
  } else {
    // element i of block blk is (j_a, i_b) with i = blk*n + j_a*b + i_b
    for (int i = threadIdx.x; i < K; i += kThreads) {
      const int blk = i / n;
      const int r = i - blk * n;
      const int ja = r / b;
      const int ib = r - ja * b;
      const uint16_t* blkp = xr + blk * n;
      float acc = 0.0f;
      for (int ia = 0; ia < a; ++ia) {
        const float h = static_cast<float>(H[ia * a + ja]);
        acc = __fadd_rn(acc, __fmul_rn(signed_elem(blkp, ia * b + ib, signs, n), h));
      }
      buf[i] = acc;
    }
  }
  __syncthreads();
  // Walsh-Hadamard butterflies over i_b inside every contiguous chunk of b elements
  const int half = K / 2;
  const int hb = b / 2;
  for (int h = 1; h < b; h <<= 1) {
    for (int p = threadIdx.x; p < half; p += kThreads) {
      const int chunk = p / hb;
      const int q = p - chunk * hb;
      const int lo = chunk * b + (q / h) * (2 * h) + (q % h);
      const int hi = lo + h;
      const float u = buf[lo];
      const float w = buf[hi];
      buf[lo] = __fadd_rn(u, w);
      buf[hi] = __fsub_rn(u, w);
    }
    __syncthreads();
  }
  if (n > 1) {
    for (int i = threadIdx.x; i < K; i += kThreads) buf[i] = __fmul_rn(buf[i], inv_sqrt_n);
    __syncthreads();
  }
}

__global__ void __launch_bounds__(kThreads)
had_quant_act_generic(RotQuantArgs args) {
  extern __shared__ float buf[];
  __shared__ float red_f[kWaves];
  const int64_t row = blockIdx.x;
  const int K = static_cast<int>(args.K);
  rotate_row_to_lds(args.x + row * args.ldx, K, args.a, args.H, args.b, args.inv_sqrt_n, args.signs, buf);
  if (args.dbg) {
    for (int i = threadIdx.x; i < K; i += kThreads) args.dbg[row * K + i] = buf[i];
  }
  const bool b8 = args.bits == 8;
  const float levels = b8 ? 255.0f : 15.0f;
  uint8_t* qrow = args.q + row * (b8 ? K : K / 2);
  const int G = K / args.group;
  if (G == 1) {
    float mn = INFINITY, mx = -INFINITY;
    for (int i = threadIdx.x; i < K; i += kThreads) {
      mn = fminf(mn, buf[i]);
      mx = fmaxf(mx, buf[i]);
    }
    mn = __fmul_rn(block_min(mn, red_f), args.clip);
    mx = __fmul_rn(block_max(mx, red_f), args.clip);
    const AsymParams p = asym_params(mn, mx, levels);
    if (threadIdx.x == 0) {
      args.alpha[row] = p.alpha;
      args.beta[row] = p.mn;
    }
    if (b8) {
      for (int j = threadIdx.x; j < K; j += kThreads) qrow[j] = static_cast<uint8_t>(asym_code(buf[j], p));
      return;
    }
    for (int j = threadIdx.x; j < K / 2; j += kThreads) {
      const uint32_t c0 = asym_code(buf[2 * j], p);
      const uint32_t c1 = asym_code(buf[2 * j + 1], p);
      qrow[j] = static_cast<uint8_t>(c0 | (c1 << 4));
    }
    return;
  }
  // one wave per group
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int gs = args.group;
  for (int g = wave; g < G; g += kWaves) {
    const float* v = buf + g * gs;
    float mn = INFINITY, mx = -INFINITY;
    for (int i = lane; i < gs; i += kWave) {
      mn = fminf(mn, v[i]);
      mx = fmaxf(mx, v[i]);
    }
    mn = __fmul_rn(wave_min(mn), args.clip);
    mx = __fmul_rn(wave_max(mx), args.clip);
    const AsymParams p = asym_params(mn, mx, levels);
    if (lane == 0) {
      args.alpha[row * G + g] = p.alpha;
      args.beta[row * G + g] = p.mn;
    }
    if (b8) {
      for (int i = lane; i < gs; i += kWave) qrow[g * gs + i] = static_cast<uint8_t>(asym_code(v[i], p));
      continue;
    }
    for (int j = lane; j < gs / 2; j += kWave) {
      const uint32_t c0 = asym_code(v[2 * j], p);
      const uint32_t c1 = asym_code(v[2 * j + 1], p);
      qrow[g * (gs / 2) + j] = static_cast<uint8_t>(c0 | (c1 << 4));
    }
  }
}

__global__ void __launch_bounds__(kThreads)
pack_w4_generic(RotQuantArgs args) {
  extern __shared__ float buf[];
  __shared__ float red_f[kWaves];
  __shared__ int red_i[kWaves];
  const int64_t row = blockIdx.x;
  const int K = static_cast<int>(args.K);
  rotate_row_to_lds(args.x + row * args.ldx, K, args.a, args.H, args.b, args.inv_sqrt_n, args.signs, buf);
  float amax = 0.0f;
  for (int i = threadIdx.x; i < K; i += kThreads) amax = fmaxf(amax, fabsf(buf[i]));
  amax = block_max(amax, red_f);
  const float alpha = sym_alpha(amax);
  const float inv = __fdiv_rn(1.0f, alpha);
  uint8_t* qrow = args.q + row * (K / 2);
  int sum = 0;
  for (int j = threadIdx.x; j < K / 2; j += kThreads) {
    const int c0 = sym_code(buf[2 * j], inv);
    const int c1 = sym_code(buf[2 * j + 1], inv);
    sum += c0 + c1;
    qrow[j] = static_cast<uint8_t>((c0 & 0xF) | ((c1 & 0xF) << 4));
  }
  sum = block_sum(sum, red_i);
  if (threadIdx.x == 0) {
    args.alpha[row] = alpha;
    args.rowsum[row] = sum;
  }
}

// Unrotated rows, per-token quantization: the row stays in registers.  Each thread owns
// chunks of 8 consecutive elements (one 16-byte load, one 4-byte (4-bit) or 8-byte (8-bit)
// code store).
template <int W, int CHMAX>
__global__ void __launch_bounds__(64 * W)
quant_rows_identity(RotQuantArgs args) {
  constexpr int T = 64 * W;
  __shared__ float red[2 * W];
  const int64_t row = blockIdx.x;
  const int nchunk = static_cast<int>(args.K / 8);
  const uint16_t* __restrict__ xr = args.x + row * args.ldx;
  float v[CHMAX][8];
  float mn = INFINITY, mx = -INFINITY;
  // every chunk load is issued before any is used (clamped index; the duplicates are not
  // counted), so a row costs one memory round trip
  uint4 dch[CHMAX];
#pragma unroll
  for (int j = 0; j < CHMAX; ++j) {
    const int ch = threadIdx.x + j * T;
    dch[j] = reinterpret_cast<const uint4*>(xr)[ch < nchunk ? ch : nchunk - 1];
  }
#pragma unroll
  for (int j = 0; j < CHMAX; ++j) {
    const int ch = threadIdx.x + j * T;
    if (ch < nchunk) {
      const uint4 d = dch[j];
      const uint32_t w[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[j][2 * i] = h2f(static_cast<uint16_t>(w[i] & 0xFFFFu));
        v[j][2 * i + 1] = h2f(static_cast<uint16_t>(w[i] >> 16));
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        mn = fminf(mn, v[j][i]);
        mx = fmaxf(mx, v[j][i]);
      }
    }
  }
  mn = wave_min(mn);
  mx = wave_max(mx);
  const int wave = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) {
    red[wave] = mn;
    red[W + wave] = mx;
  }
  __syncthreads();
  mn = red[0];
  mx = red[W];
#pragma unroll
  for (int i = 1; i < W; ++i) {
    mn = fminf(mn, red[i]);
    mx = fmaxf(mx, red[W + i]);
  }
  const bool b8 = args.bits == 8;
  const AsymParams p = asym_params(__fmul_rn(mn, args.clip), __fmul_rn(mx, args.clip), b8 ? 255.0f : 15.0f);
  if (threadIdx.x == 0) {
    args.alpha[row] = p.alpha;
    args.beta[row] = p.mn;
  }
  uint32_t* qrow = reinterpret_cast<uint32_t*>(args.q + row * (b8 ? args.K : args.K / 2));
#pragma unroll
  for (int j = 0; j < CHMAX; ++j) {
    const int ch = threadIdx.x + j * T;
    if (ch < nchunk) {
      // eq. 1's t = (v - mn) * inv, rounded after each step and clamped to [0, L] (t leaves
      // that range only with a clipped range, or by 3 ulp at the top); v_cvt_pk_u8_f32 then
      // rounds half to even, so its byte is clamp(rint(t), 0, L).  4-bit: even positions go
      // to ev, odd ones to od, and ev | od << 4 is the nibble-packed word.
      if (b8) {  // one code per byte: positions 0-3, then 4-7
        uint32_t w0 = 0, w1 = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          w0 = __builtin_amdgcn_cvt_pk_u8_f32(asym_t(v[j][i], p), i, w0);
          w1 = __builtin_amdgcn_cvt_pk_u8_f32(asym_t(v[j][4 + i], p), i, w1);
        }
        reinterpret_cast<uint2*>(qrow)[ch] = make_uint2(w0, w1);
      } else {
        uint32_t ev = 0, od = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          ev = __builtin_amdgcn_cvt_pk_u8_f32(asym_t(v[j][2 * i], p), i, ev);
          od = __builtin_amdgcn_cvt_pk_u8_f32(asym_t(v[j][2 * i + 1], p), i, od);
        }
        qrow[ch] = ev | (od << 4);
      }
      if (args.dbg) {
#pragma unroll
        for (int i = 0; i < 8; ++i) args.dbg[row * args.K + ch * 8 + i] = v[j][i];
      }
    }
  }
}

hipError_t launch_generic(void (*kern)(RotQuantArgs), const RotQuantArgs& a, hipStream_t stream) {
  const size_t lds = static_cast<size_t>(a.K) * sizeof(float);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
  if (e != hipSuccess) return e;
  return launch(kern, dim3(static_cast<unsigned>(a.rows)), dim3(kThreads), static_cast<uint32_t>(lds), stream, a);
}

}  // namespace

hipError_t launch_had_quant_act(const RotQuantArgs& a, hipStream_t stream) {
  if (a.a == 1 && a.b == 1 && a.group == a.K && a.signs == nullptr) {
    // chunks of 8 per thread sized to K, so that the registers (and with them the
    // resident workgroups per CU) follow the row length
    const dim3 grid(static_cast<unsigned>(a.rows));
    const int64_t nch = a.K / 8;
    if (nch <= 256 * 2) return launch(quant_rows_identity<4, 2>, grid, dim3(256), 0, stream, a);
    if (nch <= 256 * 4) return launch(quant_rows_identity<4, 4>, grid, dim3(256), 0, stream, a);
    if (nch <= 512 * 4) return launch(quant_rows_identity<8, 4>, grid, dim3(512), 0, stream, a);
    return launch(quant_rows_identity<8, 8>, grid, dim3(512), 0, stream, a);
  }
  const hipError_t e = launch_had_quant_kron(a, stream);
  if (e != hipErrorNotSupported) return e;
  return launch_generic(had_quant_act_generic, a, stream);
}

hipError_t launch_pack_w4(const RotQuantArgs& a, hipStream_t stream) {
  return launch_generic(pack_w4_generic, a, stream);
}

}  // namespace sq
