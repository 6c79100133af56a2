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
//   * q . c_t: v_dot2_f32_f16 on code pairs made fp16 (exact): nibbles 0, 2, 4 and 6 of a
//     code word as 1024 + c, nibbles 1, 3, 5 and 7 in place as 1024 + 16 c (five VALU per
//     word: one shift, four and-or), minus 1024 times the lane's query sums, the second part
//     divided by 16; the four lanes of a token add their parts (DPP quad permutes).
//   * Online softmax in base 2 (log2 e is folded into the scale) with one running maximum m
//     per wave (the batch maximum by DPP row rotations and permlane swaps; a rescale only
//     when it grows).  Each lane sums, over the tokens it sees, l = sum_t p_t,
//     acc_d = sum_t p_t alpha_t (1024 + c_td), or (1024 + 16 c_td) for the odd dims
//     (v_fma_mix_f32 on the same fp16 code pairs), pa = sum_t p_t alpha_t and
//     bsum = sum_t p_t beta_t; dim d is acc_d - 1024 pa (divided by 16 for odd d) + bsum.
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

// allreduce over the 16 token slots of a wave: the lanes with the same lane % 4
template <typename Op>
__device__ __forceinline__ float slots_reduce(float v, Op op) {
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

// The lane's 32 query dims (32 qd .. 32 qd + 31 of the head whose query row is qrow) as fp16
// pairs (8c + k, 8c + k + 4) matching the code pairs, the head's query sum (over the quad of
// lanes) and the code offsets of the lane's even and odd pairs (1024 times their query sums).
struct QueryPairs {
  v2h qp[4][4];
  float qsum, bias_even, bias_odd;
};
__device__ __forceinline__ void load_query(const uint16_t* qrow, int qd, QueryPairs& qq) {
  float qsum_lane = 0.0f, qodd_lane = 0.0f;  // all 32 dims; the odd dims
  const v4u* qv = reinterpret_cast<const v4u*>(qrow + 32 * qd);
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
    for (int k = 0; k < 4; ++k) qq.qp[c][k] = v2h{e[k], e[k + 4]};
#pragma unroll
    for (int k = 0; k < 8; ++k) qsum_lane = __fadd_rn(qsum_lane, static_cast<float>(e[k]));
#pragma unroll
    for (int k = 1; k < 8; k += 2) qodd_lane = __fadd_rn(qodd_lane, static_cast<float>(e[k]));
  }
  float qsum = __fadd_rn(qsum_lane, quad_xor<1>(qsum_lane));
  qq.qsum = __fadd_rn(qsum, quad_xor<2>(qsum));
  qq.bias_even = __fmul_rn(1024.0f, __fsub_rn(qsum_lane, qodd_lane));
  qq.bias_odd = __fmul_rn(1024.0f, qodd_lane);
}

// Code-word to fp16 pairs: (e0,e4) and (e2,e6) as 1024 + c, (e1,e5) and (e3,e7) as
// 1024 + 16 c (those nibbles stay in place, in mantissa bits 4-7): one shift and four and-or.
// The masks are kept in registers (a VOP3 and-or takes no literal operands).
struct PairMasks {
  uint32_t lo = 0x000F000Fu, hi = 0x00F000F0u, base = 0x64006400u;
  __device__ __forceinline__ PairMasks() { asm volatile("" : "+v"(lo), "+v"(hi), "+v"(base)); }
  __device__ __forceinline__ void pairs(uint32_t cw, v2h (&pr)[4]) const {
    const uint32_t sh = cw >> 8;
    pr[0] = __builtin_bit_cast(v2h, (cw & lo) | base);
    pr[1] = __builtin_bit_cast(v2h, (cw & hi) | base);
    pr[2] = __builtin_bit_cast(v2h, (sh & lo) | base);
    pr[3] = __builtin_bit_cast(v2h, (sh & hi) | base);
  }
};

// q . c over the lane's 32 dims of one token (code words cw), before the quad sum
__device__ __forceinline__ float lane_dot(const QueryPairs& qq, const PairMasks& pm, const v4u& cw) {
  float s0 = 0.0f, s1 = 0.0f;  // pairs 0 and 2 (1024 + c), pairs 1 and 3 (1024 + 16 c)
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    v2h pr[4];
    pm.pairs(cw[c], pr);  // dims 8c .. 8c+7 of the lane
    s0 = __builtin_amdgcn_fdot2(qq.qp[c][0], pr[0], s0, false);
    s1 = __builtin_amdgcn_fdot2(qq.qp[c][1], pr[1], s1, false);
    s0 = __builtin_amdgcn_fdot2(qq.qp[c][2], pr[2], s0, false);
    s1 = __builtin_amdgcn_fdot2(qq.qp[c][3], pr[3], s1, false);
  }
  return __fmaf_rn(__fsub_rn(s1, qq.bias_odd), 0.0625f, __fsub_rn(s0, qq.bias_even));
}

// acc_d += pa (1024 + c_d) (odd d: 1024 + 16 c_d) over the lane's 32 dims of one token
__device__ __forceinline__ void lane_accumulate(float (&acc)[32], float pa, const PairMasks& pm, const v4u& cw) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    v2h pr[4];
    pm.pairs(cw[c], pr);
#pragma unroll
    for (int k = 0; k < 4; ++k) {  // pair k holds dims 8c + k and 8c + k + 4
      acc[8 * c + k] = __fmaf_rn(pa, static_cast<float>(pr[k][0]), acc[8 * c + k]);
      acc[8 * c + k + 4] = __fmaf_rn(pa, static_cast<float>(pr[k][1]), acc[8 * c + k + 4]);
    }
  }
}

// Partial attention state of one wave: running maximum m (base 2), and per lane the sums
// over the tokens it has seen: l = sum p, acc_d = sum p alpha (1024 + c_d), pa = sum p alpha,
// bsum = sum p beta.
struct WaveAttn {
  float m = -INFINITY, l = 0.0f, bsum = 0.0f, pa_sum = 0.0f;
  float acc[32];
};

// One wave's pass over the batches first, first + step, ... (count of them) of 16 tokens of
// head (b, h); lane l = 4 tok + qd.
template <bool P16>
__device__ __forceinline__ void attend(const AttnArgs& a, int64_t b, int64_t h, int first, int step, int count,
                                       WaveAttn& st) {
  const int lane = threadIdx.x & 63;
  const int tok = lane >> 2;
  const int qd = lane & 3;
  const int64_t S = a.S;
  QueryPairs qq;
  load_query(a.q + (b * a.H + h) * 128, qd, qq);
  const PairMasks pm;

  // ---- cache of this (batch, head): token t at byte t * H * 64 (codes) / t * H * 4 (scales)
  const int64_t row0 = b * S * a.H + h;
  const int64_t cspan = ((S - 1) * a.H + 1) * 64;
  const __amdgpu_buffer_rsrc_t rk = rsrc(a.kq + row0 * 64, cspan);
  const __amdgpu_buffer_rsrc_t rv = rsrc(a.vq + row0 * 64, cspan);
  const void* pb = qd == 0 ? a.ka : qd == 1 ? a.kb : qd == 2 ? a.va : a.vb;  // this lane's scale array
  // token offsets fit 32 bits: S * H * 64 < 2^31 is checked on the host
  const uint32_t H32 = static_cast<uint32_t>(a.H), S32 = static_cast<uint32_t>(S);
  const uint32_t cstride = H32 * 64;

  v4u kc[kDepth], vc[kDepth];
  float pv[kDepth];
  auto load = [&](int slot, int it) {
    const uint32_t t = static_cast<uint32_t>(first + step * it) * 16 + tok;
    const bool ok = it < count && t < S32;  // else codes out of range (zeros), scale of token 0
    const uint32_t co = ok ? t * cstride + 16 * qd : 0x80000000u;
    kc[slot] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rk, co, 0, 0));
    vc[slot] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rv, co, 0, 0));
    const int64_t pi = row0 + (ok ? t * H32 : 0u);
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

#pragma unroll
  for (int d = 0; d < kDepth; ++d) load(d, d);
  for (int it0 = 0; it0 < count; it0 += kDepth) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      const int it = it0 + d;
      const uint32_t t = static_cast<uint32_t>(first + step * it) * 16 + tok;
      const bool ok = it < count && t < S32;  // uniform over the quad of a token
      // q . c_t over the lane's 32 dims, then over the quad
      float dot = lane_dot(qq, pm, kc[d]);
      dot = __fadd_rn(dot, quad_xor<1>(dot));
      dot = __fadd_rn(dot, quad_xor<2>(dot));
      const float ka = quad_bcast<0>(pv[d]), kb = quad_bcast<1>(pv[d]);
      const float va = quad_bcast<2>(pv[d]), vb = quad_bcast<3>(pv[d]);
      const float s = ok ? __fmul_rn(cs, __fmaf_rn(ka, dot, __fmul_rn(kb, qq.qsum))) : -INFINITY;
      const float mb = slots_reduce(s, [](float u, float v) { return fmaxf(u, v); });
      if (mb > m) {  // (uniform) new running maximum: rescale the sums
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
        lane_accumulate(acc, pa, pm, vc[d]);
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

// Dim e of a lane's 32 from its sum acc_e: the code offset (1024 pa) removed, the odd
// dims' codes (1024 + 16 c) scaled back by 1/16 (exact), the betas added.
__device__ __forceinline__ float dim_value(float acc, float off, float bsum, int e) {
  const float v = __fsub_rn(acc, off);
  return __fadd_rn(e & 1 ? __fmul_rn(v, 0.0625f) : v, bsum);
}

// The token slots of a head share m: their sums add up (every lane ends with its head's
// totals of its 32 dims).
__device__ __forceinline__ void wave_total(WaveAttn& st) {
  auto add = [](float u, float v) { return __fadd_rn(u, v); };
  st.l = slots_reduce(st.l, add);
  st.bsum = slots_reduce(st.bsum, add);
  st.pa_sum = slots_reduce(st.pa_sum, add);
#pragma unroll
  for (int e = 0; e < 32; ++e) st.acc[e] = slots_reduce(st.acc[e], add);
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
    for (int e = 0; e < 32; ++e) red_acc[w][32 * qd + e] = dim_value(acc[e], off, bsum, e);
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

// ---- split over the sequence (flash-decoding): workgroup (b, 16-head group g, chunk c) of 8
// waves.  Lane l = 4 hh + qd serves head 16 g + hh, dims 32 qd .. 32 qd + 31, so one load of
// the wave brings the 1 KB of codes of one token for the group's 16 heads (half of a 32-head
// token line), and the four parameter loads 64 contiguous bytes each.  The chunk's tokens go
// one per wave and step (wave w takes token 8 i + w of the chunk, so the 8 waves walk the
// chunk's lines together), two tokens in flight (94 VGPRs).  On [8, 2048, 32, 128] this
// measured 20.4 us against 22.8 us for batches of 4 tokens (154 VGPRs) and 21.0-21.3 us
// with 3 or 4 in flight.  Each lane keeps its head's state; a batch's scores are in the
// lane, so its maximum (and the rare rescale) needs no cross-lane step.  The 8 waves merge in LDS; each head leaves its
// partial state (m, l, the 128 dims with the code offset removed and the betas added) in
// part, and the combine kernel merges the chunks of a head.
// FINAL (a single chunk): the workgroup divides and stores the output itself.
// LDS row of a head's 128 dims in the merge: four quarters of 32, each padded to 36 floats,
// so that the 16-byte stores of lanes 4 hh + qd (16 of them at a time) and the merge's reads
// meet no bank conflicts (with rows of 128 floats all 16 heads' lanes of one quarter hit the
// same banks: 9e5 conflict cycles per launch)
constexpr int kQuarter = 36;
constexpr int kDimRow = 4 * kQuarter;

template <int WAVES>
constexpr int part_lds_bytes() {
  return WAVES * kAttnGroupHeads * (kDimRow + 2) * 4;
}

// WAVES waves of batches of TB tokens (a chunk is made of WAVES x TB-token batches), DEPTH
// batches in flight per wave, at least WPE waves per SIMD.
template <bool P16, bool FINAL, int kSplitWaves = kAttnSplitWaves, int kBatch = kAttnBatch, int WPE = 2,
          int kDepth = kAttnDepth>
__global__ void __launch_bounds__(64 * kSplitWaves, WPE)
attn_decode_part(AttnArgs a) {
  constexpr int kChunkUnit = kSplitWaves * kBatch;
  // dynamic LDS (part_lds_bytes bytes): the waves' dims [wave][head][kDimRow], then (m, l) [wave][head]
  extern __shared__ __attribute__((aligned(16))) float split_lds[];
  auto red_d = reinterpret_cast<float (*)[kAttnGroupHeads][kDimRow]>(split_lds);
  auto red_ml = reinterpret_cast<float (*)[kAttnGroupHeads][2]>(split_lds + kSplitWaves * kAttnGroupHeads * kDimRow);
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int hh = lane >> 2, qd = lane & 3;
  // the workgroup count (B * chunks * NG, at most B * NG or about the CUs) fits 32 bits
  const int NG = static_cast<int>((a.H + kAttnGroupHeads - 1) / kAttnGroupHeads), NC = static_cast<int>(a.chunks);
  // Workgroups go round-robin over the 8 XCDs.  When the count allows, the NG head groups of
  // one (batch, chunk) get ids equal mod 8, so they run on one XCD and the two halves of a
  // token's parameter lines (64 bytes each of a 128-byte line) come through one L2.
  const int id = static_cast<int>(blockIdx.x), total = static_cast<int>(gridDim.x);
  int g, bc;
  if (NG > 1 && total % (8 * NG) == 0) {
    g = (id / 8) % NG;
    bc = (id / (8 * NG)) * 8 + id % 8;
  } else {
    g = id % NG;
    bc = id / NG;
  }
  const int c = bc % NC;
  const int64_t b = bc / NC;
  const int64_t h = kAttnGroupHeads * g + hh;
  const bool hok = h < a.H;
  const int64_t hq = hok ? h : a.H - 1;  // lanes past the heads run on the last head and store nothing
  QueryPairs qq;
  load_query(a.q + (b * a.H + hq) * 128, qd, qq);
  const PairMasks pm;

  // tokens of the chunk: units of kChunkUnit tokens first .. first + count - 1; wave w,
  // batch i: tokens kChunkUnit (first + i) + kBatch w + j, j < kBatch
  const int nb = static_cast<int>((a.S + kChunkUnit - 1) / kChunkUnit);
  const int first = c * static_cast<int>(a.chunk_batches);
  const int count = min(static_cast<int>(a.chunk_batches), nb - first);
  const uint32_t H32 = static_cast<uint32_t>(a.H), S32 = static_cast<uint32_t>(a.S);
  // token offsets fit 32 bits: S * H * 64 < 2^31 is checked on the host
  const int64_t row0 = b * a.S * a.H;
  const __amdgpu_buffer_rsrc_t rk = rsrc(a.kq + row0 * 64, a.S * a.H * 64);
  const __amdgpu_buffer_rsrc_t rv = rsrc(a.vq + row0 * 64, a.S * a.H * 64);
  const void* pb = qd == 0 ? a.ka : qd == 1 ? a.kb : qd == 2 ? a.va : a.vb;  // this lane's scale array

  v4u kc[kDepth][kBatch], vc[kDepth][kBatch];
  float pv[kDepth][kBatch];
  auto token = [&](int i, int j) { return static_cast<uint32_t>(kChunkUnit * (first + i) + kBatch * w + j); };
  auto load = [&](int buf, int i) {
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const uint32_t t = token(i, j);
      const bool ok = hok && i < count && t < S32;  // else codes out of range (zeros), scale of token 0
      const uint32_t co = ok ? (t * H32 + static_cast<uint32_t>(h)) * 64 + 16 * qd : 0x80000000u;
      kc[buf][j] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rk, co, 0, 0));
      vc[buf][j] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rv, co, 0, 0));
      const int64_t pi = row0 + (ok ? t * H32 + static_cast<uint32_t>(h) : 0u);
      if constexpr (P16)
        pv[buf][j] = h2f(static_cast<const uint16_t*>(pb)[pi]);
      else
        pv[buf][j] = static_cast<const float*>(pb)[pi];
    }
  };

  float m = -INFINITY, l = 0.0f, bsum = 0.0f, pa_sum = 0.0f;
  float acc[32];
#pragma unroll
  for (int e = 0; e < 32; ++e) acc[e] = 0.0f;
  const float cs = a.scale_log2e;
  auto process = [&](int buf, int i) {
    float sc[kBatch];
    float mb = -INFINITY;
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const bool ok = hok && i < count && token(i, j) < S32;  // uniform over the quad
      float dot = lane_dot(qq, pm, kc[buf][j]);
      dot = __fadd_rn(dot, quad_xor<1>(dot));
      dot = __fadd_rn(dot, quad_xor<2>(dot));
      const float ka = quad_bcast<0>(pv[buf][j]), kb = quad_bcast<1>(pv[buf][j]);
      sc[j] = ok ? __fmul_rn(cs, __fmaf_rn(ka, dot, __fmul_rn(kb, qq.qsum))) : -INFINITY;
      mb = fmaxf(mb, sc[j]);
    }
    if (mb > m) {  // new running maximum of this lane's head: rescale the sums
      const float f = rescale(m, mb);
      l = __fmul_rn(l, f);
      bsum = __fmul_rn(bsum, f);
      pa_sum = __fmul_rn(pa_sum, f);
#pragma unroll
      for (int e = 0; e < 32; ++e) acc[e] = __fmul_rn(acc[e], f);
      m = mb;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (sc[j] != -INFINITY) {
        const float va = quad_bcast<2>(pv[buf][j]), vb = quad_bcast<3>(pv[buf][j]);
        const float p = exp2f(__fsub_rn(sc[j], m));
        l = __fadd_rn(l, p);
        bsum = __fmaf_rn(p, vb, bsum);
        const float pa = __fmul_rn(p, va);
        pa_sum = __fadd_rn(pa_sum, pa);
        lane_accumulate(acc, pa, pm, vc[buf][j]);
      }
    }
  };
#pragma unroll
  for (int d = 0; d < kDepth; ++d) load(d, d);
  for (int i = 0; i < count; i += kDepth) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      process(d, i + d);
      load(d, i + d + kDepth);
    }
  }

  // the waves' states of each head meet in LDS
  const float off = __fmul_rn(1024.0f, pa_sum);
  if (qd == 0) {
    red_ml[w][hh][0] = m;
    red_ml[w][hh][1] = l;
  }
  float4* rd = reinterpret_cast<float4*>(&red_d[w][hh][kQuarter * qd]);
#pragma unroll
  for (int e = 0; e < 32; e += 4)
    rd[e / 4] = make_float4(dim_value(acc[e], off, bsum, e), dim_value(acc[e + 1], off, bsum, e + 1),
                            dim_value(acc[e + 2], off, bsum, e + 2), dim_value(acc[e + 3], off, bsum, e + 3));
  __syncthreads();
  // item x of 512: head x / 32 of the group, dims 4 (x % 32) .. + 3
  for (int x = threadIdx.x; x < 32 * kAttnGroupHeads; x += 64 * kSplitWaves) {
    const int mh = x >> 5, md = 4 * (x & 31);
    const int64_t oh = kAttnGroupHeads * g + mh;
    if (oh >= a.H) break;  // the heads past H come last; no barrier follows
    float M = -INFINITY;
#pragma unroll
    for (int v = 0; v < kSplitWaves; ++v) M = fmaxf(M, red_ml[v][mh][0]);
    float L = 0.0f, D0 = 0.0f, D1 = 0.0f, D2 = 0.0f, D3 = 0.0f;
#pragma unroll
    for (int v = 0; v < kSplitWaves; ++v) {
      const float f = rescale(red_ml[v][mh][0], M);  // 0 for a wave that saw no token
      const float4 d = *reinterpret_cast<const float4*>(&red_d[v][mh][kQuarter * (md / 32) + md % 32]);
      L = __fmaf_rn(red_ml[v][mh][1], f, L);
      D0 = __fmaf_rn(d.x, f, D0);
      D1 = __fmaf_rn(d.y, f, D1);
      D2 = __fmaf_rn(d.z, f, D2);
      D3 = __fmaf_rn(d.w, f, D3);
    }
    if constexpr (FINAL) {  // a chunk holds every token (L > 0: S >= 1)
      uint32_t* o = reinterpret_cast<uint32_t*>(a.out + (b * a.H + oh) * 128 + md);
      o[0] = static_cast<uint32_t>(f2h(__fdiv_rn(D0, L))) | (static_cast<uint32_t>(f2h(__fdiv_rn(D1, L))) << 16);
      o[1] = static_cast<uint32_t>(f2h(__fdiv_rn(D2, L))) | (static_cast<uint32_t>(f2h(__fdiv_rn(D3, L))) << 16);
    } else {
      float* pr = a.part + ((b * a.H + oh) * NC + c) * kAttnPart;
      if (md == 0) {
        pr[0] = M;
        pr[1] = L;
      }
      *reinterpret_cast<float4*>(pr + 4 + md) = make_float4(D0, D1, D2, D3);
    }
  }
}

// One wave per head: the chunks' states (at most 64) rescaled to their common maximum and
// summed.  Lane c holds chunk c's maximum and sum; the dims (lane l finishes 2 l and 2 l + 1)
// come 32 chunks at a time, added in chunk order.  Every load of a pass is issued before the
// first is used, at clamped chunk indices (a chunk past NC gets weight 0), so the maxima,
// the sums and the first 32 chunks' dims take one round trip together.  One wave per
// workgroup, so the heads spread over all CUs (0.2-0.3 us less than four waves per
// workgroup on [8, 2048, 32, 128]).
__global__ void __launch_bounds__(64)
attn_decode_combine(AttnArgs a) {
  const int lane = threadIdx.x;
  const int64_t x = blockIdx.x;  // B * H < 2^31 is checked on the host
  const int NC = static_cast<int>(a.chunks);
  const float* pr = a.part + x * NC * kAttnPart;
  const int cl = lane < NC ? lane : NC - 1;
  const float2 ml = *reinterpret_cast<const float2*>(pr + cl * kAttnPart);
  float2 d[32];
#pragma unroll
  for (int j = 0; j < 32; ++j) d[j] = reinterpret_cast<const float2*>(pr + min(j, NC - 1) * kAttnPart + 4)[lane];
  const float mc = lane < NC ? ml.x : -INFINITY;
  const float lc = lane < NC ? ml.y : 0.0f;
  float M = mc;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  const float fc = rescale(mc, M);  // 0 for lanes past the chunks
  float L = __fmul_rn(lc, fc);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) L = __fadd_rn(L, __shfl_xor(L, o));
  float A0 = 0.0f, A1 = 0.0f;
  auto add32 = [&](int c0) {
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const float f = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(fc), c0 + j));
      A0 = __fmaf_rn(d[j].x, f, A0);
      A1 = __fmaf_rn(d[j].y, f, A1);
    }
  };
  add32(0);
  if (NC > 32) {  // chunks 32 .. 63
#pragma unroll
    for (int j = 0; j < 32; ++j)
      d[j] = reinterpret_cast<const float2*>(pr + min(32 + j, NC - 1) * kAttnPart + 4)[lane];
    add32(32);
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

namespace {
template <bool P16, bool FINAL>
hipError_t launch_part(const AttnArgs& a, unsigned parts, hipStream_t stream) {
  constexpr auto kern = attn_decode_part<P16, FINAL>;
  constexpr int lds = part_lds_bytes<kAttnSplitWaves>();
  const hipError_t init = set_max_lds<kern>(lds);  // above the 64 KB default
  if (init != hipSuccess) return init;
  return launch(kern, dim3(parts), dim3(64 * kAttnSplitWaves), lds, stream, a);
}
}  // namespace

hipError_t launch_attn_decode_split(const AttnArgs& a, hipStream_t stream) {
  const int64_t NG = (a.H + kAttnGroupHeads - 1) / kAttnGroupHeads;
  const unsigned parts = static_cast<unsigned>(a.B * a.chunks * NG);
  if (a.chunks == 1)
    return a.param16 ? launch_part<true, true>(a, parts, stream) : launch_part<false, true>(a, parts, stream);
  hipError_t e = a.param16 ? launch_part<true, false>(a, parts, stream) : launch_part<false, false>(a, parts, stream);
  if (e != hipSuccess) return e;
  return launch(attn_decode_combine, dim3(static_cast<unsigned>(a.B * a.H)), dim3(64), 0, stream, a);
}

hipError_t launch_attn_decode_kv4(const AttnArgs& a, hipStream_t stream) {
  const unsigned blocks = static_cast<unsigned>(a.B * a.H);
  return a.param16 ? launch(attn_decode_kv4<true>, dim3(blocks), dim3(kThreads), 0, stream, a)
                   : launch(attn_decode_kv4<false>, dim3(blocks), dim3(kThreads), 0, stream, a);
}

}  // namespace sq
