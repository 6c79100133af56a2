// Decode attention over the 4-bit K/V cache written by the R3 + KV4 kernel: the step that
// consumes it.  R3 is orthonormal, so the rotated query against the rotated keys gives the
// scores of the unrotated pair (Sec. 3.1); keys and values are dequantised by eq. 1 group by
// group, K_t = alpha_t c_t + beta_t.  For each (batch, head):
//     out = softmax_t(scale * q . K_t) V,
//     q . K_t = alpha_t (q . c_t) + beta_t sum(q).
//
// One workgroup of 8 waves per (batch, head).  Batch i of 16 cached tokens goes to wave
// i % 8; lane l = 4 tok + qd holds token tok of the batch and head dims 32 qd .. 32 qd + 31,
// i.e. one 16-byte load of K codes and one of V codes (a batch reads 16 x 64 contiguous
// bytes of each), plus the token's four scales.
//   * q . c_t: v_dot2_f32_f16 on code pairs made fp16 as 1024 + c (exact), minus 1024 times
//     the lane's query sum; the four lanes of a token add their parts (DPP quad permutes).
//   * Each lane keeps an online softmax over the tokens it sees, in base 2 (log2 e is folded
//     into the scale): running maximum m, sum l, and acc_d = sum_t p_t alpha_t c_td,
//     bsum = sum_t p_t beta_t for its 32 dims.
//   * At the end the 16 token slots of a wave merge by butterflies over the lane index, and
//     the 8 waves in LDS; out_d = (acc_d + bsum) / l.
// Workgroup i serves head index x(i) = (i % 8) * (G / 8) + i / 8 when the G = B * H heads
// are a multiple of 8: workgroups go round-robin over the 8 XCDs, so heads h and h + 1 (the
// two 64-byte halves of a 128-byte line of a token) are read through the same L2.
#include "sq_device.h"
#include "sq_internal.h"

namespace sq {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kDepth = 4;  // batches in flight per wave

typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, static_cast<int>(bytes), 0x00020000);
}

template <int M>
__device__ __forceinline__ float quad_xor(float v) {
  constexpr int ctrl = (M == 1) ? 0xB1 : 0x4E;  // quad_perm [1,0,3,2] / [2,3,0,1]
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), ctrl, 0xF, 0xF, false));
}

// 2^(a - b), 0 when a is -inf (an empty partial state)
__device__ __forceinline__ float rescale(float a, float b) {
  return a == -INFINITY ? 0.0f : exp2f(__fsub_rn(a, b));
}

__global__ void __launch_bounds__(kThreads)
attn_decode_kv4(AttnArgs a) {
  __shared__ float red_ml[kWaves][3];
  __shared__ float red_acc[kWaves][128];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int tok = lane >> 2;
  const int qd = lane & 3;
  const int64_t G = a.B * a.H;
  const int64_t i = blockIdx.x;
  const int64_t x = (G % 8 == 0) ? (i % 8) * (G / 8) + i / 8 : i;
  const int64_t b = x / a.H, h = x % a.H;
  const int64_t S = a.S;

  // ---- query: the lane's 32 dims as fp16 pairs (8w+e, 8w+e+4) matching the code pairs
  v2h qp[4][4];
  float qsum_lane = 0.0f;
  {
    const v4u* qv = reinterpret_cast<const v4u*>(a.q + (b * a.H + h) * 128 + 32 * qd);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const v4u v = qv[c];  // dims 32 qd + 8 c .. + 7: words [q0|q1] [q2|q3] [q4|q5] [q6|q7]
      _Float16 e[8];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        e[2 * k] = __builtin_bit_cast(_Float16, static_cast<uint16_t>(v[k] & 0xFFFFu));
        e[2 * k + 1] = __builtin_bit_cast(_Float16, static_cast<uint16_t>(v[k] >> 16));
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) qp[c][k] = v2h{e[k], e[k + 4]};
#pragma unroll
      for (int k = 0; k < 8; ++k) qsum_lane = __fadd_rn(qsum_lane, static_cast<float>(e[k]));
    }
  }
  float qsum = __fadd_rn(qsum_lane, quad_xor<1>(qsum_lane));
  qsum = __fadd_rn(qsum, quad_xor<2>(qsum));
  const float bias1024 = __fmul_rn(1024.0f, qsum_lane);

  // ---- cache of this (batch, head): token t at byte t * H * 64 (codes) / t * H * 4 (scales)
  const int64_t row0 = b * S * a.H + h;
  const int64_t cspan = ((S - 1) * a.H + 1) * 64, sspan = ((S - 1) * a.H + 1) * 4;
  const __amdgpu_buffer_rsrc_t rk = rsrc(a.kq + row0 * 64, cspan);
  const __amdgpu_buffer_rsrc_t rv = rsrc(a.vq + row0 * 64, cspan);
  const __amdgpu_buffer_rsrc_t rka = rsrc(a.ka + row0, sspan);
  const __amdgpu_buffer_rsrc_t rkb = rsrc(a.kb + row0, sspan);
  const __amdgpu_buffer_rsrc_t rva = rsrc(a.va + row0, sspan);
  const __amdgpu_buffer_rsrc_t rvb = rsrc(a.vb + row0, sspan);
  const uint32_t cstride = static_cast<uint32_t>(a.H * 64), sstride = static_cast<uint32_t>(a.H * 4);

  const int nb = static_cast<int>((S + 15) / 16);  // batches of 16 tokens
  const int mine = nb > w ? (nb - w + kWaves - 1) / kWaves : 0;
  v4u kc[kDepth], vc[kDepth];
  float ka[kDepth], kb[kDepth], va[kDepth], vb[kDepth];
  auto load = [&](int slot, int it) {
    const int64_t t = static_cast<int64_t>(w + kWaves * it) * 16 + tok;
    const bool ok = it < mine && t < S;  // past the end: out of range, reads zeros
    const uint32_t co = ok ? static_cast<uint32_t>(t) * cstride + 16 * qd : 0x80000000u;
    const uint32_t so = ok ? static_cast<uint32_t>(t) * sstride : 0x80000000u;
    kc[slot] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rk, co, 0, 0));
    vc[slot] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rv, co, 0, 0));
    ka[slot] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rka, so, 0, 0));
    kb[slot] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rkb, so, 0, 0));
    va[slot] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rva, so, 0, 0));
    vb[slot] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rvb, so, 0, 0));
  };

  float m = -INFINITY, l = 0.0f, bsum = 0.0f;
  float acc[32];
#pragma unroll
  for (int d = 0; d < 32; ++d) acc[d] = 0.0f;
  const float cs = a.scale_log2e;

#pragma unroll
  for (int d = 0; d < kDepth; ++d) load(d, d);
  for (int it0 = 0; it0 < mine; it0 += kDepth) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      const int it = it0 + d;
      const int64_t t = static_cast<int64_t>(w + kWaves * it) * 16 + tok;
      const bool ok = it < mine && t < S;  // uniform over the quad of a token
      // q . c_t over the lane's 32 dims, then over the quad
      float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t cw = kc[d][c];  // dims 8c .. 8c+7 of the lane: nibbles e = 0..7
        const uint32_t pA = (cw & 0x000F000Fu) | 0x64006400u;          // (e0, e4)
        const uint32_t pB = ((cw >> 4) & 0x000F000Fu) | 0x64006400u;   // (e1, e5)
        const uint32_t pC = ((cw >> 8) & 0x000F000Fu) | 0x64006400u;   // (e2, e6)
        const uint32_t pD = ((cw >> 12) & 0x000F000Fu) | 0x64006400u;  // (e3, e7)
        s0 = __builtin_amdgcn_fdot2(qp[c][0], __builtin_bit_cast(v2h, pA), s0, false);
        s1 = __builtin_amdgcn_fdot2(qp[c][1], __builtin_bit_cast(v2h, pB), s1, false);
        s0 = __builtin_amdgcn_fdot2(qp[c][2], __builtin_bit_cast(v2h, pC), s0, false);
        s1 = __builtin_amdgcn_fdot2(qp[c][3], __builtin_bit_cast(v2h, pD), s1, false);
      }
      float dot = __fsub_rn(__fadd_rn(s0, s1), bias1024);
      dot = __fadd_rn(dot, quad_xor<1>(dot));
      dot = __fadd_rn(dot, quad_xor<2>(dot));
      const float s = __fmul_rn(cs, __fmaf_rn(ka[d], dot, __fmul_rn(kb[d], qsum)));
      if (ok) {
        if (s > m) {  // new running maximum: rescale what has been summed
          const float f = rescale(m, s);
          l = __fmul_rn(l, f);
          bsum = __fmul_rn(bsum, f);
#pragma unroll
          for (int e = 0; e < 32; ++e) acc[e] = __fmul_rn(acc[e], f);
          m = s;
        }
        const float p = exp2f(__fsub_rn(s, m));
        l = __fadd_rn(l, p);
        bsum = __fmaf_rn(p, vb[d], bsum);
        const float pa = __fmul_rn(p, va[d]);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const uint32_t cw = vc[d][c];
          const uint32_t lo = cw & 0x0F0F0F0Fu, hi = (cw >> 4) & 0x0F0F0F0Fu;  // even / odd dims
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            acc[8 * c + 2 * k] = __fmaf_rn(pa, static_cast<float>((lo >> (8 * k)) & 0xFFu), acc[8 * c + 2 * k]);
            acc[8 * c + 2 * k + 1] = __fmaf_rn(pa, static_cast<float>((hi >> (8 * k)) & 0xFFu), acc[8 * c + 2 * k + 1]);
          }
        }
      }
      load(d, it + kDepth);
    }
  }

  // ---- the 16 token slots of the wave (lane bits 2..5) merge
#pragma unroll
  for (int off = 4; off < 64; off <<= 1) {
    const float mo = __shfl_xor(m, off, 64);
    const float lo_ = __shfl_xor(l, off, 64);
    const float bo = __shfl_xor(bsum, off, 64);
    const float mn = fmaxf(m, mo);
    const float f = rescale(m, mn), fo = rescale(mo, mn);
    l = __fmaf_rn(l, f, __fmul_rn(lo_, fo));
    bsum = __fmaf_rn(bsum, f, __fmul_rn(bo, fo));
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      const float ao = __shfl_xor(acc[e], off, 64);
      acc[e] = __fmaf_rn(acc[e], f, __fmul_rn(ao, fo));
    }
    m = mn;
  }
  if (lane < 4) {
#pragma unroll
    for (int e = 0; e < 32; ++e) red_acc[w][32 * qd + e] = acc[e];
    if (lane == 0) {
      red_ml[w][0] = m;
      red_ml[w][1] = l;
      red_ml[w][2] = bsum;
    }
  }
  __syncthreads();
  if (w != 0) return;
  // ---- the 8 waves merge; lane handles dims 2 lane, 2 lane + 1
  float M = -INFINITY;
#pragma unroll
  for (int v = 0; v < kWaves; ++v) M = fmaxf(M, red_ml[v][0]);
  float L = 0.0f, Bs = 0.0f, A0 = 0.0f, A1 = 0.0f;
#pragma unroll
  for (int v = 0; v < kWaves; ++v) {
    const float f = rescale(red_ml[v][0], M);
    L = __fmaf_rn(red_ml[v][1], f, L);
    Bs = __fmaf_rn(red_ml[v][2], f, Bs);
    A0 = __fmaf_rn(red_acc[v][2 * lane], f, A0);
    A1 = __fmaf_rn(red_acc[v][2 * lane + 1], f, A1);
  }
  const float o0 = __fdiv_rn(__fadd_rn(A0, Bs), L), o1 = __fdiv_rn(__fadd_rn(A1, Bs), L);
  reinterpret_cast<uint32_t*>(a.out + (b * a.H + h) * 128)[lane] =
      static_cast<uint32_t>(f2h(o0)) | (static_cast<uint32_t>(f2h(o1)) << 16);
}

}  // namespace

hipError_t launch_attn_decode_kv4(const AttnArgs& a, hipStream_t stream) {
  const unsigned blocks = static_cast<unsigned>(a.B * a.H);
  return launch(attn_decode_kv4, dim3(blocks), dim3(kThreads), 0, stream, a);
}

}  // namespace sq
