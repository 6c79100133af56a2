// Decode attention over the 4-bit K/V cache written by the R3 + KV4 kernel: the step that
// consumes it.  R3 is orthonormal, so the rotated query against the rotated keys gives the
// scores of the unrotated pair (Sec. 3.1); keys and values are dequantised by eq. 1 group by
// group, K_t = alpha_t c_t + beta_t.  For each (batch, head):
//     out = softmax_t(scale * q . K_t) V,
//     q . K_t = alpha_t (q . c_t) + beta_t sum(q).
//
// One workgroup of 16 waves (four per SIMD, to hide HBM latency) per (batch, head).
// Batch i of 16 cached tokens goes to wave i % 16; lane l = 4 tok + qd holds token tok of
// the batch and head dims 32 qd .. 32 qd + 31, i.e. one 16-byte load of K codes and one of
// V codes (a batch reads 16 x 64 contiguous bytes of each); lane qd of the token loads its
// scale number qd (k_alpha, k_beta, v_alpha, v_beta) and the quad shares them by DPP.
//   * q . c_t: v_dot2_f32_f16 on code pairs made fp16 as 1024 + c (exact), minus 1024 times
//     the lane's query sum; the four lanes of a token add their parts (DPP quad permutes).
//   * Online softmax in base 2 (log2 e is folded into the scale) with one running maximum m
//     per wave (the batch maximum by DPP row rotations and permlane swaps; a rescale only
//     when it grows).  Each lane sums, over the tokens it sees, l = sum_t p_t,
//     acc_d = sum_t p_t alpha_t (1024 + c_td) (v_fma_mix_f32 on the same fp16 code pairs),
//     pa = sum_t p_t alpha_t and bsum = sum_t p_t beta_t; dim d is acc_d - 1024 pa + bsum.
//   * At the end the 16 token slots of a wave add up in registers (same maximum), and the 16
//     waves merge in LDS; out_d = (sum of the waves' rescaled dims) / (their rescaled l).
// The group parameters are fp32, or fp16 (P16: half the parameter bytes of the cache).
// Workgroup i serves head index x(i) = (i % 8) * (G / 8) + i / 8 when the G = B * H heads
// are a multiple of 8: workgroups go round-robin over the 8 XCDs, so heads h and h + 1 (the
// two 64-byte halves of a 128-byte line of a token) are read through the same L2.
#include <mutex>

#include "sq_device.h"
#include "sq_internal.h"

namespace sq {
namespace {

constexpr int kWaves = 16;
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

// allreduce over the token slots of a wave: the lanes with the same lane % 4 (HPW = 1, 16
// slots) or lane % 8 (HPW = 2, 8 slots)
template <int HPW = 1, typename Op>
__device__ __forceinline__ float slots_reduce(float v, Op op) {
  if constexpr (HPW == 1)
    v = op(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x124, 0xF, 0xF, false)));  // row_ror:4
  v = op(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128, 0xF, 0xF, false)));  // row_ror:8
  const bool odd_row = (threadIdx.x >> 4) & 1, upper = (threadIdx.x >> 5) & 1;
  const auto s16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = op(v, __uint_as_float(odd_row ? s16[0] : s16[1]));  // the other row of the 32-lane half
  const auto s32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = op(v, __uint_as_float(upper ? s32[0] : s32[1]));    // the other half
  return v;
}

// value of lane L of this lane's quad
template <int L>
__device__ __forceinline__ float quad_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), L * 0x55, 0xF, 0xF, false));
}

// 2^(a - b), 0 when a is -inf (an empty partial state)
__device__ __forceinline__ float rescale(float a, float b) {
  return a == -INFINITY ? 0.0f : exp2f(__fsub_rn(a, b));
}

// Partial attention state of one wave: running maximum m (base 2), and per lane the sums
// over the tokens it has seen: l = sum p, acc_d = sum p alpha (1024 + c_d), pa = sum p alpha,
// bsum = sum p beta.
struct WaveAttn {
  float m = -INFINITY, l = 0.0f, bsum = 0.0f, pa_sum = 0.0f;
  float acc[32];
};

// One wave's pass over the batches first, first + step, ... (count of them) of 16 / HPW
// tokens.  HPW = 1: every lane serves head (b, h); lane l = 4 tok + qd.  HPW = 2: the wave
// serves heads h and h + 1 (one 128-byte piece of a token's line), lane l = 8 tok + 4 hp + qd
// serves head h + hp; when h + 1 is past the heads, its lanes see no tokens.
template <bool P16, int HPW = 1>
__device__ __forceinline__ void attend(const AttnArgs& a, int64_t b, int64_t h0, int first, int step, int count,
                                       WaveAttn& st) {
  static_assert(HPW == 1 || HPW == 2, "one or two heads per wave");
  constexpr int TS = 16 / HPW;  // tokens per batch
  const int lane = threadIdx.x & 63;
  const int tok = lane >> (HPW == 2 ? 3 : 2);
  const int hp = HPW == 2 ? (lane >> 2) & 1 : 0;
  const int qd = lane & 3;
  const int64_t S = a.S;
  const int nh = HPW == 2 && h0 + 1 < a.H ? 2 : 1;  // heads of this wave
  const bool hok = hp < nh;
  const int64_t h = h0 + (hok ? hp : 0);             // this lane's head
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
  const int64_t row0 = b * S * a.H + h0;
  const int64_t cspan = ((S - 1) * a.H + nh) * 64;
  const __amdgpu_buffer_rsrc_t rk = rsrc(a.kq + row0 * 64, cspan);
  const __amdgpu_buffer_rsrc_t rv = rsrc(a.vq + row0 * 64, cspan);
  const void* pb = qd == 0 ? a.ka : qd == 1 ? a.kb : qd == 2 ? a.va : a.vb;  // this lane's scale array
  // token offsets fit 32 bits: S * H * 64 < 2^31 is checked on the host
  const uint32_t H32 = static_cast<uint32_t>(a.H), S32 = static_cast<uint32_t>(S);
  const uint32_t cstride = H32 * 64;

  v4u kc[kDepth], vc[kDepth];
  float pv[kDepth];
  auto load = [&](int slot, int it) {
    const uint32_t t = static_cast<uint32_t>(first + step * it) * TS + tok;
    const bool ok = hok && it < count && t < S32;  // else codes out of range (zeros), scale of token 0
    const uint32_t co = ok ? t * cstride + 64 * hp + 16 * qd : 0x80000000u;
    kc[slot] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rk, co, 0, 0));
    vc[slot] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rv, co, 0, 0));
    const int64_t pi = row0 + (ok ? t * H32 + hp : 0u);
    if constexpr (P16)
      pv[slot] = h2f(static_cast<const uint16_t*>(pb)[pi]);
    else
      pv[slot] = static_cast<const float*>(pb)[pi];
  };

  float m = st.m, l = st.l, bsum = st.bsum, pa_sum = st.pa_sum;
  float acc[32];
#pragma unroll
  for (int d = 0; d < 32; ++d) acc[d] = st.acc[d];
  const float cs = a.scale_log2e;
  // code pair masks kept in registers (a VOP3 and-or takes no literal operands)
  uint32_t kMask = 0x000F000Fu, kBase = 0x64006400u;
  asm volatile("" : "+v"(kMask), "+v"(kBase));
  // the four fp16 pairs (1024 + c) of a code word: (e0,e4) (e1,e5) (e2,e6) (e3,e7)
  auto pairs = [&](uint32_t cw, v2h (&pr)[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) pr[k] = __builtin_bit_cast(v2h, ((cw >> (4 * k)) & kMask) | kBase);
  };

#pragma unroll
  for (int d = 0; d < kDepth; ++d) load(d, d);
  for (int it0 = 0; it0 < count; it0 += kDepth) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      const int it = it0 + d;
      const uint32_t t = static_cast<uint32_t>(first + step * it) * TS + tok;
      const bool ok = hok && it < count && t < S32;  // uniform over the quad of a token
      // q . c_t over the lane's 32 dims, then over the quad
      float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        v2h pr[4];
        pairs(kc[d][c], pr);  // dims 8c .. 8c+7 of the lane
        s0 = __builtin_amdgcn_fdot2(qp[c][0], pr[0], s0, false);
        s1 = __builtin_amdgcn_fdot2(qp[c][1], pr[1], s1, false);
        s0 = __builtin_amdgcn_fdot2(qp[c][2], pr[2], s0, false);
        s1 = __builtin_amdgcn_fdot2(qp[c][3], pr[3], s1, false);
      }
      float dot = __fsub_rn(__fadd_rn(s0, s1), bias1024);
      dot = __fadd_rn(dot, quad_xor<1>(dot));
      dot = __fadd_rn(dot, quad_xor<2>(dot));
      const float ka = quad_bcast<0>(pv[d]), kb = quad_bcast<1>(pv[d]);
      const float va = quad_bcast<2>(pv[d]), vb = quad_bcast<3>(pv[d]);
      const float s = ok ? __fmul_rn(cs, __fmaf_rn(ka, dot, __fmul_rn(kb, qsum))) : -INFINITY;
      const float mb = slots_reduce<HPW>(s, [](float u, float v) { return fmaxf(u, v); });
      if (mb > m) {  // (uniform over a head's lanes) new running maximum: rescale the sums
        const float f = rescale(m, mb);
        l = __fmul_rn(l, f);
        bsum = __fmul_rn(bsum, f);
        pa_sum = __fmul_rn(pa_sum, f);
#pragma unroll
        for (int e = 0; e < 32; ++e) acc[e] = __fmul_rn(acc[e], f);
        m = mb;
      }
      if (ok) {
        const float p = exp2f(__fsub_rn(s, m));
        l = __fadd_rn(l, p);
        bsum = __fmaf_rn(p, vb, bsum);
        const float pa = __fmul_rn(p, va);
        pa_sum = __fadd_rn(pa_sum, pa);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          v2h pr[4];
          pairs(vc[d][c], pr);
#pragma unroll
          for (int k = 0; k < 4; ++k) {  // pair k holds dims 8c + k and 8c + k + 4
            acc[8 * c + k] = __fmaf_rn(pa, static_cast<float>(pr[k][0]), acc[8 * c + k]);
            acc[8 * c + k + 4] = __fmaf_rn(pa, static_cast<float>(pr[k][1]), acc[8 * c + k + 4]);
          }
        }
      }
      load(d, it + kDepth);
    }
  }
  st.m = m;
  st.l = l;
  st.bsum = bsum;
  st.pa_sum = pa_sum;
#pragma unroll
  for (int d = 0; d < 32; ++d) st.acc[d] = acc[d];
}

// The token slots of a head share m: their sums add up (every lane ends with its head's
// totals of its 32 dims).
template <int HPW = 1>
__device__ __forceinline__ void wave_total(WaveAttn& st) {
  auto add = [](float u, float v) { return __fadd_rn(u, v); };
  st.l = slots_reduce<HPW>(st.l, add);
  st.bsum = slots_reduce<HPW>(st.bsum, add);
  st.pa_sum = slots_reduce<HPW>(st.pa_sum, add);
#pragma unroll
  for (int e = 0; e < 32; ++e) st.acc[e] = slots_reduce<HPW>(st.acc[e], add);
}

template <bool P16>
__global__ void __launch_bounds__(kThreads)
attn_decode_kv4(AttnArgs a) {
  __shared__ float red_ml[kWaves][2];
  __shared__ float red_acc[kWaves][128];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int qd = lane & 3;
  const int64_t G = a.B * a.H;
  const int64_t i = blockIdx.x;
  const int64_t x = (G % 8 == 0) ? (i % 8) * (G / 8) + i / 8 : i;
  const int64_t b = x / a.H, h = x % a.H;
  const int nb = static_cast<int>((a.S + 15) / 16);  // batches of 16 tokens
  const int mine = nb > w ? (nb - w + kWaves - 1) / kWaves : 0;
  WaveAttn st;
#pragma unroll
  for (int d = 0; d < 32; ++d) st.acc[d] = 0.0f;
  attend<P16>(a, b, h, w, kWaves, mine, st);
  wave_total(st);
  const float m = st.m, l = st.l, bsum = st.bsum, pa_sum = st.pa_sum;
  const float* acc = st.acc;

  // remove the 1024 offset of the code pairs and add the betas: the wave's dims
  const float off = __fmul_rn(1024.0f, pa_sum);
  if (lane < 4) {
#pragma unroll
    for (int e = 0; e < 32; ++e) red_acc[w][32 * qd + e] = __fadd_rn(__fsub_rn(acc[e], off), bsum);
    if (lane == 0) {
      red_ml[w][0] = m;
      red_ml[w][1] = l;
    }
  }
  __syncthreads();
  if (w != 0) return;
  // ---- the 16 waves merge; lane handles dims 2 lane, 2 lane + 1
  float M = -INFINITY;
#pragma unroll
  for (int v = 0; v < kWaves; ++v) M = fmaxf(M, red_ml[v][0]);
  float L = 0.0f, A0 = 0.0f, A1 = 0.0f;
#pragma unroll
  for (int v = 0; v < kWaves; ++v) {
    const float f = rescale(red_ml[v][0], M);
    L = __fmaf_rn(red_ml[v][1], f, L);
    A0 = __fmaf_rn(red_acc[v][2 * lane], f, A0);
    A1 = __fmaf_rn(red_acc[v][2 * lane + 1], f, A1);
  }
  const float o0 = __fdiv_rn(A0, L), o1 = __fdiv_rn(A1, L);
  reinterpret_cast<uint32_t*>(a.out + (b * a.H + h) * 128)[lane] =
      static_cast<uint32_t>(f2h(o0)) | (static_cast<uint32_t>(f2h(o1)) << 16);
}

// ---- split over the sequence (flash-decoding): workgroup (b, chunk c, group g of 32
// heads) of 16 waves; wave w serves heads 32 g + 2 w and 32 g + 2 w + 1 over the chunk's
// batches of 8 tokens, so each of its loads brings whole 128-byte lines (8 tokens x 128
// bytes), where one wave per head uses half of every line it touches, and the workgroup
// reads whole 2 KB token lines of a 32-head cache.  Each head leaves its partial state (m,
// l, the 128 dims with the code offset removed and the betas added) in part; the combine
// kernel merges the chunks of a head.
// FINAL (a single chunk): the lanes divide and store the output themselves.
constexpr int kSplitWaves = kAttnGroupHeads / 2;

template <bool P16, bool FINAL>
__global__ void __launch_bounds__(64 * kSplitWaves, 4)
attn_decode_part(AttnArgs a) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int qd = lane & 3;
  const int hp = (lane >> 2) & 1;
  // the workgroup count (B * chunks * NG, at most B * NG or about four times the CUs) fits 32 bits
  const int NG = static_cast<int>((a.H + kAttnGroupHeads - 1) / kAttnGroupHeads), NC = static_cast<int>(a.chunks);
  const int g = static_cast<int>(blockIdx.x) % NG;
  const int c = (static_cast<int>(blockIdx.x) / NG) % NC;
  const int b = static_cast<int>(blockIdx.x) / NG / NC;
  const int h0 = kAttnGroupHeads * g + 2 * w;
  if (h0 >= a.H) return;  // no workgroup barrier follows
  const int nb = static_cast<int>((a.S + 7) / 8);  // batches of 8 tokens
  const int first = 2 * c * static_cast<int>(a.chunk_batches);
  const int count = min(2 * static_cast<int>(a.chunk_batches), nb - first);
  WaveAttn st;
#pragma unroll
  for (int d = 0; d < 32; ++d) st.acc[d] = 0.0f;
  attend<P16, 2>(a, b, h0, first, 1, count, st);
  wave_total<2>(st);
  const int h = h0 + hp;
  if (lane >= 8 || h >= a.H) return;  // lanes 4 hp + qd of token slot 0 write
  const float off = __fmul_rn(1024.0f, st.pa_sum);
  float* dims = st.acc;  // in place: the lane's 32 dims
#pragma unroll
  for (int e = 0; e < 32; ++e) dims[e] = __fadd_rn(__fsub_rn(st.acc[e], off), st.bsum);
  if constexpr (FINAL) {  // a chunk holds every token (l > 0: S >= 1)
    uint32_t* o = reinterpret_cast<uint32_t*>(a.out + (static_cast<int64_t>(b) * a.H + h) * 128 + 32 * qd);
#pragma unroll
    for (int e = 0; e < 32; e += 2)
      o[e / 2] = static_cast<uint32_t>(f2h(__fdiv_rn(dims[e], st.l))) |
                 (static_cast<uint32_t>(f2h(__fdiv_rn(dims[e + 1], st.l))) << 16);
  } else {
    float* pr = a.part + ((static_cast<int64_t>(b) * a.H + h) * NC + c) * kAttnPart;
    if (qd == 0) {
      pr[0] = st.m;
      pr[1] = st.l;
    }
    float4* pd = reinterpret_cast<float4*>(pr + 4 + 32 * qd);
#pragma unroll
    for (int e = 0; e < 8; ++e) pd[e] = make_float4(dims[4 * e], dims[4 * e + 1], dims[4 * e + 2], dims[4 * e + 3]);
  }
}

// One wave per head: the chunks' states (at most 64) rescaled to their common maximum and
// summed.  Lane c holds chunk c's maximum and sum; the dims (lane l finishes 2 l and 2 l + 1)
// are loaded 32 chunks at a time, all 32 loads in flight together, and added in chunk
// order.
__global__ void __launch_bounds__(256)
attn_decode_combine(AttnArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t x = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (x >= a.B * a.H) return;
  const int NC = static_cast<int>(a.chunks);
  const float* pr = a.part + x * NC * kAttnPart;
  const float mc = lane < NC ? pr[lane * kAttnPart] : -INFINITY;
  const float lc = lane < NC ? pr[lane * kAttnPart + 1] : 0.0f;
  float M = mc;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  const float fc = rescale(mc, M);  // 0 for lanes past the chunks
  float L = __fmul_rn(lc, fc);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) L = __fadd_rn(L, __shfl_xor(L, o));
  float A0 = 0.0f, A1 = 0.0f;
  for (int c0 = 0; c0 < NC; c0 += 32) {
    float2 d[32];
#pragma unroll
    for (int j = 0; j < 32; ++j)
      d[j] = c0 + j < NC ? reinterpret_cast<const float2*>(pr + (c0 + j) * kAttnPart + 4)[lane] : float2{0.0f, 0.0f};
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const float f = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(fc), min(c0 + j, 63)));
      A0 = __fmaf_rn(d[j].x, f, A0);
      A1 = __fmaf_rn(d[j].y, f, A1);
    }
  }
  reinterpret_cast<uint32_t*>(a.out + x * 128)[lane] =
      static_cast<uint32_t>(f2h(__fdiv_rn(A0, L))) | (static_cast<uint32_t>(f2h(__fdiv_rn(A1, L))) << 16);
}

// Partial states of the allocation-free split attention: one array per device, kept until
// the process ends.  Host code uses its device address from hipGetSymbolAddress, never
// the array's name.
static __device__ __align__(256) unsigned char scratch[kAttnScratchBytes];

}  // namespace

hipError_t attn_scratch(void** ptr) {
  static std::mutex mu;
  static void* addr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {  // once per device, with that device current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_attn_decode_split(const AttnArgs& a, hipStream_t stream) {
  const int64_t NG = (a.H + kAttnGroupHeads - 1) / kAttnGroupHeads;
  const unsigned parts = static_cast<unsigned>(a.B * a.chunks * NG);
  const dim3 block(64 * kSplitWaves);
  if (a.chunks == 1)
    return a.param16 ? launch(attn_decode_part<true, true>, dim3(parts), block, 0, stream, a)
                     : launch(attn_decode_part<false, true>, dim3(parts), block, 0, stream, a);
  hipError_t e = a.param16 ? launch(attn_decode_part<true, false>, dim3(parts), block, 0, stream, a)
                           : launch(attn_decode_part<false, false>, dim3(parts), block, 0, stream, a);
  if (e != hipSuccess) return e;
  const unsigned heads = static_cast<unsigned>((a.B * a.H + 3) / 4);
  return launch(attn_decode_combine, dim3(heads), dim3(256), 0, stream, a);
}

hipError_t launch_attn_decode_kv4(const AttnArgs& a, hipStream_t stream) {
  const unsigned blocks = static_cast<unsigned>(a.B * a.H);
  return a.param16 ? launch(attn_decode_kv4<true>, dim3(blocks), dim3(kThreads), 0, stream, a)
                   : launch(attn_decode_kv4<false>, dim3(blocks), dim3(kThreads), 0, stream, a);
}

}  // namespace sq
