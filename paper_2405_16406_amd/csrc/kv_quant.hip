// R3 on post-RoPE Q and K (Sec. 3.1) fused with 4-bit (or, for the KV8 setting, 8-bit)
// asymmetric K/V cache quantization.
//
// One head vector (D = 128 fp16) is one quantization group.  Four lanes (a quad) own a
// group; lane j of the quad holds the 32 elements i = 32*k + 8*j + e (k = 0..3, e = 0..7),
// i.e. four 16-byte chunks, so each 16-byte load or store instruction of a wave covers
// whole 64-byte lines (16 groups x 64 bytes).  The 128-point Walsh-Hadamard transform is
// five in-register butterfly stages (index bits 0-2 and 5-6) and two cross-lane stages
// (bits 3-4: quad lanes xor 1 and xor 2, by DPP quad permutes, no LDS); min/max reduce
// in registers and then across the quad the same way.  Codes are made bytes by
// v_cvt_pk_u8_f32, which rounds half to even like rint, and nibble-packed.
//   V (the quantizer input itself): rint(fl(fl(v - mn) * fl(1/alpha))), eq. 1 step by step.
//   K (rotated, 1/sqrt(128) folded into alpha and beta): rint(fma(v, 1/alpha, -mn/alpha));
//     this can move a code by one only where the value sits on a rounding boundary, which
//     the rotated path allows anyway.
// A clipping ratio r in (0, 1] per cache (App. A "Quantization choice") quantizes each
// group's range [r min, r max]; the code argument is clamped to [0, L] before the
// conversion (which by itself saturates at 255 only), so values outside take the end codes.
// P16 stores alpha and beta as fp16: the fp32 pair (of the reported values) rounded to
// nearest with saturation, a zero fp16 alpha making the group constant, and the codes taken
// from the stored pair (V: fl(fl(v - beta16) * fl(1/alpha16)) as eq. 1's steps; K: one fma
// in the unscaled domain).
#include "sq_device.h"
#include "sq_internal.h"

#include <type_traits>

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kD = 128;

typedef unsigned v4u __attribute__((ext_vector_type(4)));

// value of the lane whose quad index is this lane's xor M (M = 1 or 2)
template <int M>
__device__ __forceinline__ float quad_xor(float v) {
  constexpr int ctrl = (M == 1) ? 0xB1 : 0x4E;  // quad_perm [1,0,3,2] / [2,3,0,1]
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), ctrl, 0xF, 0xF, false));
}

// the lane's four 16-byte chunks of a group: chunk k holds elements 32*k + 8*j .. + 7
__device__ __forceinline__ void load_raw(const uint16_t* __restrict__ grp_base, int j, v4u (&raw)[4]) {
#pragma unroll
  for (int k = 0; k < 4; ++k) raw[k] = *reinterpret_cast<const v4u*>(grp_base + 32 * k + 8 * j);
}

// e[8*k + q] = element 32*k + 8*j + q of the group (fp16 -> fp32, exact)
__device__ __forceinline__ void widen(const v4u (&raw)[4], float (&e)[32]) {
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      e[8 * k + 2 * i] = h2f(static_cast<uint16_t>(raw[k][i] & 0xFFFFu));
      e[8 * k + 2 * i + 1] = h2f(static_cast<uint16_t>(raw[k][i] >> 16));
    }
}

__device__ __forceinline__ void bfly(float& lo, float& hi) {
  const float u = lo, w = hi;
  lo = __fadd_rn(u, w);
  hi = __fsub_rn(u, w);
}

// unscaled 128-point Sylvester transform of the group held by the quad
__device__ __forceinline__ void fwht128(float (&e)[32], int j) {
  // register index r = 8*k + q: bits 0-2 of r are element bits 0-2, bits 3-4 are bits 5-6
#pragma unroll
  for (int h = 1; h < 32; h <<= 1)
#pragma unroll
    for (int r = 0; r < 32; ++r)
      if ((r & h) == 0) bfly(e[r], e[r + h]);
  // element bits 3 and 4 live in the quad lane index: lower partner u + w, upper w - u
  const float s1 = (j & 1) ? -1.0f : 1.0f;
#pragma unroll
  for (int r = 0; r < 32; ++r) e[r] = __fmaf_rn(s1, e[r], quad_xor<1>(e[r]));
  const float s2 = (j & 2) ? -1.0f : 1.0f;
#pragma unroll
  for (int r = 0; r < 32; ++r) e[r] = __fmaf_rn(s2, e[r], quad_xor<2>(e[r]));
}

// eq. 1 asymmetric codes of the quad's group; `scale` multiplies the reported alpha and beta
// (1 when e holds the values themselves, and then the codes follow eq. 1 step by step).
// 4-bit: element 32*k + 8*j + q -> nibble of byte 16*k + 4*j + q/2 of the group's 64 bytes;
// 8-bit: -> byte 32*k + 8*j + q of its 128 bytes.
template <bool EXACT, int BITS, bool P16>
__device__ __forceinline__ void quant_store(const float (&e)[32], int j, float scale, float clip, int64_t grp,
                                            uint8_t* q, void* alpha, void* beta) {
  float mn = e[0], mx = e[0];
#pragma unroll
  for (int r = 1; r < 32; ++r) {
    mn = fminf(mn, e[r]);
    mx = fmaxf(mx, e[r]);
  }
  mn = fminf(mn, quad_xor<1>(mn));
  mx = fmaxf(mx, quad_xor<1>(mx));
  mn = __fmul_rn(fminf(mn, quad_xor<2>(mn)), clip);
  mx = __fmul_rn(fmaxf(mx, quad_xor<2>(mx)), clip);
  constexpr float kL = BITS == 8 ? 255.0f : 15.0f;
  // alpha of the reported (scaled) values decides the constant-group case
  const float r_u = __fsub_rn(mx, mn);
  const float a_u = __fdiv_rn(r_u, kL);
  const float a_s = __fmul_rn(a_u, scale);
  float inv, nb, mn_t = mn;  // code argument: fma(v, inv, nb), or (v - mn_t) * inv (EXACT)
  uint16_t a16 = 0, b16 = 0;
  bool cst;
  if constexpr (P16) {
    a16 = f2h_sat(a_s);
    cst = a_s < kMinNormal || (a16 & 0x7FFFu) == 0;
    if (cst) a16 = 0x3C00u;  // 1.0
    b16 = f2h_sat(__fmul_rn(mn, scale));
    const float inv16 = __fdiv_rn(1.0f, h2f(a16));
    mn_t = h2f(b16);  // EXACT: scale is 1
    inv = EXACT ? inv16 : __fmul_rn(scale, inv16);
    nb = -__fmul_rn(mn_t, inv16);
  } else {
    cst = a_s < kMinNormal;
    inv = cst ? 1.0f : __fdiv_rn(1.0f, a_u);
    nb = -__fmul_rn(mn, inv);
  }
  uint8_t* qg = q + grp * (kD * BITS / 8);
  if constexpr (BITS == 8) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      uint32_t w[2] = {0u, 0u};
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        const float v = e[8 * k + x];
        const float t = EXACT ? __fmul_rn(__fsub_rn(v, mn_t), inv) : __fmaf_rn(v, inv, nb);
        w[x >> 2] = __builtin_amdgcn_cvt_pk_u8_f32(__builtin_amdgcn_fmed3f(t, 0.0f, kL), x & 3, w[x >> 2]);
      }
      *reinterpret_cast<uint2*>(qg + 32 * k + 8 * j) = make_uint2(w[0], w[1]);
    }
  }
#pragma unroll
  for (int k = 0; k < (BITS == 8 ? 0 : 4); ++k) {
    // bytes of the 8 codes q = 0..7, then even codes low nibble, odd codes high nibble
    uint32_t ev = 0, od = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float t0, t1;
      if constexpr (EXACT) {
        t0 = __fmul_rn(__fsub_rn(e[8 * k + 2 * i], mn_t), inv);
        t1 = __fmul_rn(__fsub_rn(e[8 * k + 2 * i + 1], mn_t), inv);
      } else {
        t0 = __fmaf_rn(e[8 * k + 2 * i], inv, nb);
        t1 = __fmaf_rn(e[8 * k + 2 * i + 1], inv, nb);
      }
      // rounds half to even
      ev = __builtin_amdgcn_cvt_pk_u8_f32(__builtin_amdgcn_fmed3f(t0, 0.0f, kL), i, ev);
      od = __builtin_amdgcn_cvt_pk_u8_f32(__builtin_amdgcn_fmed3f(t1, 0.0f, kL), i, od);
    }
    *reinterpret_cast<uint32_t*>(qg + 16 * k + 4 * j) = ev | (od << 4);
  }
  if (j == 0) {
    if constexpr (P16) {
      static_cast<uint16_t*>(alpha)[grp] = a16;
      static_cast<uint16_t*>(beta)[grp] = b16;
    } else {
      static_cast<float*>(alpha)[grp] = cst ? 1.0f : a_s;
      static_cast<float*>(beta)[grp] = __fmul_rn(mn, scale);
    }
  }
}

// EARLY: the three head vectors are requested before any is transformed (the outputs could
// alias the inputs as far as the compiler knows, so it would not move these loads up by
// itself).  That takes 97 VGPRs (4 waves per SIMD); it pays when the grid has more
// workgroups than that occupancy holds, and otherwise each vector is loaded just before its
// transform.
template <bool EARLY, int BITS, bool P16>
__global__ void __launch_bounds__(kThreads)
qk_had_kvquant_v2(KvArgs a) {
  const int64_t grp = (static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x) / 4;
  const int j = threadIdx.x & 3;
  if (grp >= a.groups) return;  // the 4 lanes of a group leave together
  const int64_t base = grp * kD;
  v4u rq[4], rk[4], rv[4];
  load_raw(a.q + base, j, rq);
  if constexpr (EARLY) {
    load_raw(a.k + base, j, rk);
    load_raw(a.v + base, j, rv);
  }
  float e[32];

  // Q: rotate, scale, fp16
  widen(rq, e);
  fwht128(e, j);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v4u o;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      o[i] = static_cast<uint32_t>(f2h(__fmul_rn(e[8 * k + 2 * i], a.inv_sqrt_d))) |
             (static_cast<uint32_t>(f2h(__fmul_rn(e[8 * k + 2 * i + 1], a.inv_sqrt_d))) << 16);
    *reinterpret_cast<v4u*>(a.q_rot + base + 32 * k + 8 * j) = o;
  }

  // K: rotate, quantize with the 1/sqrt(128) scale folded into alpha and beta
  if constexpr (!EARLY) load_raw(a.k + base, j, rk);
  widen(rk, e);
  fwht128(e, j);
  if (a.dbg_k) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int q = 0; q < 8; ++q) a.dbg_k[base + 32 * k + 8 * j + q] = __fmul_rn(e[8 * k + q], a.inv_sqrt_d);
  }
  quant_store<false, BITS, P16>(e, j, a.inv_sqrt_d, a.k_clip, grp, a.kq, a.ka, a.kb);

  // V: quantize
  if constexpr (!EARLY) load_raw(a.v + base, j, rv);
  widen(rv, e);
  quant_store<true, BITS, P16>(e, j, 1.0f, a.v_clip, grp, a.vq, a.va, a.vb);
}

}  // namespace

hipError_t launch_qk_had_kvquant(const KvArgs& a, hipStream_t stream) {
  const int64_t threads = a.groups * 4;
  const unsigned blocks = static_cast<unsigned>((threads + kThreads - 1) / kThreads);
  // Measured on MI355X: [8, 2048, 32, 128] (8192 workgroups) 112 vs 118 us with the early
  // loads; [1, 2048, 32, 128] (1024 workgroups, 4 per CU) 13.6 vs 15.1 us without them.
  const bool early = blocks >= 16 * 256;
  const dim3 grid(blocks), block(kThreads);
  auto go = [&](auto early_c, auto p16_c) -> hipError_t {
    constexpr bool E = decltype(early_c)::value, P = decltype(p16_c)::value;
    return a.bits == 8 ? launch(qk_had_kvquant_v2<E, 8, P>, grid, block, 0, stream, a)
                       : launch(qk_had_kvquant_v2<E, 4, P>, grid, block, 0, stream, a);
  };
  using T = std::true_type;
  using N = std::false_type;
  if (a.param16) return early ? go(T{}, T{}) : go(N{}, T{});
  return early ? go(T{}, N{}) : go(N{}, N{});
}

}  // namespace sq
