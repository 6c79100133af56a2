// Fast path of the online rotation + per-token 4-bit quantization for rows of length
// K = a * b rotated by (H_a (x) S_b) / sqrt(K), element i = i_a * b + i_b.
//
// View a row as X2[i_a][i_b] (a x b, i_b contiguous).  Then Y2 = H_a^T X2 S_b, computed as
// its transpose T[i_b][j_a] = (S_b^T X2^T H_a)[i_b][j_a] = y[j_a * b + i_b]:
//   * dense stage X2^T H_a on the fp16 matrix cores (v_mfma_f32_32x32x16_f16): the inputs
//     are exact fp16 and H_a is +-1, so every product is exact and only the fp32
//     accumulation rounds.  MFMA tile: M = 32 consecutive i_b, N = 32 j_a, K = 16 i_a;
//     an A fragment gathers 8 values of one column i_b at stride b (consecutive lanes
//     read consecutive i_b, so each gather is coalesced).  H_a is zero-padded to
//     APAD x (NT*32).
//   * Sylvester stage over i_b.  A 32x32 fp32 MFMA result gives lane l, register r the
//     element m = 8*(r/4) + 4*(l/32) + r%4 of column l%32: i_b bits 0, 1, 3, 4 are
//     register bits, bit 2 is the lane half, the next bits index the M tiles of a wave,
//     and the top bits the waves of the workgroup (MW of them).
//       MW == 1: bit 2 is one cross-lane exchange per value.
//       MW  > 1: after the in-register stages every lane writes its values to LDS and
//                reads back complete groups over (wave, lane half), so the remaining
//                log2(2*MW) stages are in-register too.
//   * per-row min/max, then the eq. 1 asymmetric quantizer with the 1/sqrt(K) scale
//     folded into alpha and beta: code = rint((v - mn) * (1/alpha)) in the unscaled
//     domain, rounded by adding 2^23 (exact round-half-to-even for 0 <= t < 2^22; the
//     code is then the low bits of the float).  Codes of consecutive i_b of one column
//     are nibble-packed in registers (the two lane halves swap 16-bit halves) and
//     stored straight to global memory: output position j_a * b + i_b.
// Persistent: each workgroup (MW*NW waves; waves split i_b by MW and j_a by NW) loads the
// +-1 fragments once and walks rows blockIdx.x, +gridDim.x, ..., prefetching the next
// row while it transforms the current one.
#include "sq_device.h"
#include "sq_internal.h"

#include <utility>

namespace sq {
namespace {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

template <int A, int APAD, int NT, int B, int MW, int NW, bool STAGE>
struct Kron {
  static constexpr int W = MW * NW;          // waves per workgroup
  static constexpr int THREADS = 64 * W;
  static constexpr int KS = APAD / 16;       // k-steps of the dense stage
  static constexpr int MT = B / 32 / MW;     // M tiles (32 i_b each) per wave
  static constexpr int NTW = NT / NW;        // N tiles (32 j_a each) per wave
  static constexpr int K = A * B;
  static constexpr int P = MT * 16;          // values per lane before the exchange (NTW == 1)
  static constexpr int SL = MW > 1 ? P / (2 * MW) : 0;  // positions per lane after the exchange
  static constexpr int NV = MW > 1 ? SL * 2 * MW : MT * NTW * 16;  // values per lane
  static constexpr int ROW_CHUNKS = K * 2 / 16;                    // 16-byte chunks of a row
  static constexpr int PF = STAGE ? (ROW_CHUNKS + THREADS - 1) / THREADS : 0;
  static_assert(APAD % 16 == 0 && APAD >= A && NT * 32 >= A, "padding");
  static_assert(A % 4 == 0, "Hadamard orders are multiples of 4");
  static_assert(B % (32 * MW) == 0 && NT % NW == 0, "tiling");
  static_assert(MW == 1 || (NTW == 1 && !STAGE), "wave split over i_b: one N tile, direct loads");
  static_assert(MW == 1 || (P % (2 * MW)) == 0, "exchange slices");
  static_assert(K % 16 == 0, "16-code packing");
  // LDS layout (bytes)
  static constexpr int ROW_BYTES = STAGE ? K * 2 : 0;
  static constexpr int XCH_BYTES = MW > 1 ? MW * P * 64 * 4 : 0;
  static constexpr int RED_BYTES = 2 * W * 4;
  static constexpr int LDS = ROW_BYTES + XCH_BYTES + RED_BYTES;
};

// Calls f(std::integral_constant<int, I>) for I = 0 .. N-1 (compile-time indices).
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ void bfly(float& lo, float& hi) {
  const float u = lo, w = hi;
  lo = __fadd_rn(u, w);
  hi = __fsub_rn(u, w);
}

// A fragment of the dense stage: the 8 fp16 X2[i_a][i_b] of one column i_b (colp points
// at element i_b of the row) for i_a = k0 .. k0+7, at stride B; zero for i_a >= A.
template <int A, int B>
__device__ __forceinline__ v8h gather_afrag(const uint16_t* __restrict__ colp, int k0) {
  uint32_t w[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int k = k0 + 2 * p;  // A is a multiple of 4 and k0 of 8: pairs are all in or all out
    w[p] = (k < A) ? (static_cast<uint32_t>(colp[k * B]) | (static_cast<uint32_t>(colp[(k + 1) * B]) << 16)) : 0u;
  }
  return __builtin_bit_cast(v8h, make_uint4(w[0], w[1], w[2], w[3]));
}

// rint(t) for 0 <= t < 2^22 as the low bits of t + 2^23 (one IEEE round-half-to-even add)
__device__ __forceinline__ uint32_t rne_bits(float t) {
  return __float_as_uint(__fadd_rn(t, 8388608.0f));
}

// Variant kernels (VAR): the sign flips of S (random Hadamard S H, Sec. 2.2) as the fp16
// sign-bit mask of one 16-byte chunk, from the chunk's 8 int8 entries of S (+-1: bit 7 of
// byte e is the sign of element e)
__device__ __forceinline__ v4u sign_mask(const uint2 s) {
  return v4u{((s.x << 8) & 0x8000u) | ((s.x << 16) & 0x80000000u), ((s.x >> 8) & 0x8000u) | (s.x & 0x80000000u),
             ((s.y << 8) & 0x8000u) | ((s.y << 16) & 0x80000000u), ((s.y >> 8) & 0x8000u) | (s.y & 0x80000000u)};
}
// and the code argument t clamped to [0, L], which a clipped range needs (v_cvt_pk_u8_f32
// alone saturates at 255 only)
template <bool VAR, int BITS>
__device__ __forceinline__ float code_arg(float t) {
  if constexpr (VAR) return __builtin_amdgcn_fmed3f(t, 0.0f, BITS == 8 ? 255.0f : 15.0f);
  return t;
}

template <int A, int APAD, int NT, int B, int MW, int NW, bool STAGE, bool DBG>
__global__ void __launch_bounds__(64 * MW * NW)
had_quant_kron(RotQuantArgs args) {
  using C = Kron<A, APAD, NT, B, MW, NW, STAGE>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint16_t* lds_row = reinterpret_cast<uint16_t*>(smem);
  float* lds_xch = reinterpret_cast<float*>(smem + C::ROW_BYTES);
  float* lds_red = reinterpret_cast<float*>(smem + C::ROW_BYTES + C::XCH_BYTES);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave % MW;
  const int wn = wave / MW;
  const int g = lane >> 5;
  const int c = lane & 31;
  const int64_t rows = args.rows;
  const float s_n = args.inv_sqrt_n;

  // +-1 factor as MFMA B fragments: B[k][n] = H[k][n], k = ks*16 + 8g + e, n = tile*32 + c
  v8h bfrag[C::NTW][C::KS];
#pragma unroll
  for (int nt = 0; nt < C::NTW; ++nt) {
    const int n = (wn * C::NTW + nt) * 32 + c;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = ks * 16 + 8 * g + e;
        const float h = (k < A && n < A) ? static_cast<float>(args.H[k * A + n]) : 0.0f;
        bfrag[nt][ks][e] = static_cast<_Float16>(h);
      }
    }
  }

  int64_t row = blockIdx.x;
  if (row >= rows) return;

  // first row: A fragments in registers (direct) or the row in LDS (staged)
  v8h af[STAGE ? 1 : C::MT][C::KS];
  v4u pf[STAGE ? C::PF : 1];
  auto load_direct = [&](int64_t r) {
    const uint16_t* xr = args.x + r * args.ldx;
#pragma unroll
    for (int mt = 0; mt < (STAGE ? 1 : C::MT); ++mt) {
      const int ib = (wm * C::MT + mt) * 32 + c;
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) af[mt][ks] = gather_afrag<A, B>(xr + ib, ks * 16 + 8 * g);
    }
  };
  // staged rows: chunk j of this thread is 16-byte chunk threadIdx.x + j * THREADS of the row;
  // the load index is clamped so every load is unconditional (the duplicate is not stored)
  auto load_stage = [&](int64_t r) {
    const v4u* xr = reinterpret_cast<const v4u*>(args.x + r * args.ldx);
#pragma unroll
    for (int j = 0; j < C::PF; ++j) {
      const int i = threadIdx.x + j * C::THREADS;
      pf[j] = xr[i < C::ROW_CHUNKS ? i : C::ROW_CHUNKS - 1];
    }
  };
  auto store_stage = [&]() {
#pragma unroll
    for (int j = 0; j < C::PF; ++j) {
      const int i = threadIdx.x + j * C::THREADS;
      if (i < C::ROW_CHUNKS) reinterpret_cast<v4u*>(lds_row)[i] = pf[j];
    }
  };
  if constexpr (STAGE) {
    load_stage(row);
    store_stage();
    __syncthreads();
  } else {
    load_direct(row);
  }

  for (; row < rows; row += gridDim.x) {
    const int64_t next = row + gridDim.x;
    // ---- dense stage
    v16f acc[C::MT][C::NTW];
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < C::NTW; ++nt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mt][nt][r] = 0.0f;
    if constexpr (!STAGE) {
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
          acc[mt][0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[mt][ks], bfrag[0][ks], acc[mt][0], 0, 0, 0);
      if (next < rows) load_direct(next);  // prefetch: in flight during the rest of this row
    } else {
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        v8h a_[C::MT];
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt) a_[mt] = gather_afrag<A, B>(lds_row + mt * 32 + c, ks * 16 + 8 * g);
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < C::NTW; ++nt)
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a_[mt], bfrag[nt][ks], acc[mt][nt], 0, 0, 0);
      }
      if (next < rows) load_stage(next);
    }

    // ---- Sylvester stages held in registers: i_b bits 0, 1, 3, 4 (register bits) and the tile bits
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < C::NTW; ++nt)
#pragma unroll
        for (int rb = 1; rb < 16; rb <<= 1)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if ((r & rb) == 0) {
              float lo = acc[mt][nt][r], hi = acc[mt][nt][r + rb];
              bfly(lo, hi);
              acc[mt][nt][r] = lo;
              acc[mt][nt][r + rb] = hi;
            }
#pragma unroll
    for (int tb = 1; tb < C::MT; tb <<= 1)
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt)
        if ((mt & tb) == 0)
#pragma unroll
          for (int nt = 0; nt < C::NTW; ++nt)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              float lo = acc[mt][nt][r], hi = acc[mt + tb][nt][r];
              bfly(lo, hi);
              acc[mt][nt][r] = lo;
              acc[mt + tb][nt][r] = hi;
            }

    // ---- remaining bits; val[] = this lane's values, with their (i_b, j_a) given by vpos()
    float val[C::NV];
    if constexpr (MW == 1) {
      // bit 2 across the lane halves: lower half u + w, upper half w' - u' via fma(+-1, v, partner)
      const float sg = g ? -1.0f : 1.0f;
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < C::NTW; ++nt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float v = acc[mt][nt][r];
            const float p = __shfl_xor(v, 32, 64);
            val[(mt * C::NTW + nt) * 16 + r] = __fmaf_rn(sg, v, p);
          }
    } else {
      // write (wave, position, lane half, column); read back whole (wave, half) groups
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) lds_xch[((wm * C::P) + mt * 16 + r) * 64 + lane] = acc[mt][0][r];
      __syncthreads();
      const int pbase = (wm * 2 + g) * C::SL;
#pragma unroll
      for (int t = 0; t < C::SL; ++t)
#pragma unroll
        for (int s = 0; s < MW; ++s)
#pragma unroll
          for (int h = 0; h < 2; ++h) val[(t * MW + s) * 2 + h] = lds_xch[((s * C::P) + pbase + t) * 64 + h * 32 + c];
      // butterflies over (source wave, half): index bit 0 = i_b bit 2, bits 1.. = wave bits
#pragma unroll
      for (int t = 0; t < C::SL; ++t)
#pragma unroll
        for (int hb = 1; hb < 2 * MW; hb <<= 1)
#pragma unroll
          for (int q = 0; q < 2 * MW; ++q)
            if ((q & hb) == 0) bfly(val[t * 2 * MW + q], val[t * 2 * MW + q + hb]);
    }

    // ---- per-row min/max over real columns (padded columns hold exact zeros)
    float mn = INFINITY, mx = -INFINITY;
    if constexpr (MW == 1) {
#pragma unroll
      for (int nt = 0; nt < C::NTW; ++nt) {
        float a = INFINITY, b = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            a = fminf(a, val[(mt * C::NTW + nt) * 16 + r]);
            b = fmaxf(b, val[(mt * C::NTW + nt) * 16 + r]);
          }
        if ((wn * C::NTW + nt) * 32 + c < A) {
          mn = fminf(mn, a);
          mx = fmaxf(mx, b);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < C::NV; ++i) {
        mn = fminf(mn, val[i]);
        mx = fmaxf(mx, val[i]);
      }
      if (c >= A) {
        mn = INFINITY;
        mx = -INFINITY;
      }
    }
    mn = wave_min(mn);
    mx = wave_max(mx);
    if (lane == 0) {
      lds_red[wave] = mn;
      lds_red[C::W + wave] = mx;
    }
    __syncthreads();
    mn = lds_red[0];
    mx = lds_red[C::W];
#pragma unroll
    for (int w = 1; w < C::W; ++w) {
      mn = fminf(mn, lds_red[w]);
      mx = fmaxf(mx, lds_red[C::W + w]);
    }
    // eq. 1 in the unscaled domain; reported alpha, beta carry the 1/sqrt(K) scale
    // (a group whose scaled alpha is below kMinNormal is constant: alpha 1, codes 0)
    const float r_u = __fsub_rn(mx, mn);
    const float a_u = __fdiv_rn(r_u, 15.0f);
    const bool cst = __fmul_rn(a_u, s_n) < kMinNormal;
    const float inv_u = cst ? 0.0f : __fdiv_rn(1.0f, a_u);
    if (threadIdx.x == 0) {
      args.alpha[row] = cst ? 1.0f : __fmul_rn(a_u, s_n);
      args.beta[row] = __fmul_rn(mn, s_n);
    }

    // ---- codes, nibble-packed in registers, stored at output positions j_a * B + i_b
    uint8_t* qrow = args.q + row * (C::K / 2);
    auto code = [&](float v) { return rne_bits(__fmul_rn(__fsub_rn(v, mn), inv_u)) & 0xFu; };
    if constexpr (MW == 1) {
      // lane (c, g) holds i_b = mt*32 + 8*q + 4*g + e (r = 4q + e) of column j_a: runs of 4
      // positions; the partner lane half holds the other 4 of every 8, so after swapping
      // 16-bit halves each lane half owns whole 16-byte runs (32 positions): half g stores
      // the M tiles of parity g, and a wave's stores cover 1 KB contiguously.
#pragma unroll
      for (int nt = 0; nt < C::NTW; ++nt) {
        const int ja = (wn * C::NTW + nt) * 32 + c;
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt) {
          uint32_t h16[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            uint32_t h = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float v = val[(mt * C::NTW + nt) * 16 + 4 * q + e];
              h |= code(v) << (4 * e);
              if constexpr (DBG) {
                if (ja < A) args.dbg[row * C::K + ja * B + mt * 32 + 8 * q + 4 * g + e] = __fmul_rn(v, s_n);
              }
            }
            h16[q] = h;
          }
          const uint32_t p01 = static_cast<uint32_t>(__shfl_xor(static_cast<int>(h16[0] | (h16[1] << 16)), 32, 64));
          const uint32_t p23 = static_cast<uint32_t>(__shfl_xor(static_cast<int>(h16[2] | (h16[3] << 16)), 32, 64));
          const uint32_t other[4] = {p01 & 0xFFFFu, p01 >> 16, p23 & 0xFFFFu, p23 >> 16};
          uint32_t w[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) w[q] = g ? (other[q] | (h16[q] << 16)) : (h16[q] | (other[q] << 16));
          if ((mt & 1) == g && ja < A)
            *reinterpret_cast<uint4*>(qrow + (ja * B + mt * 32) / 2) = make_uint4(w[0], w[1], w[2], w[3]);
        }
      }
    } else {
      // lane (c, u = 2*wm + g) holds, for every exchange slice s, the 2*SL consecutive
      // positions ibase + s*MT*32 + 8*(t>>2) + 4*h + (t&3) <-> val[(t*MW + s)*2 + h]
      constexpr int TPU = 16 / C::SL;  // exchange slices per 16-register tile
      static_assert(C::SL == 4 || C::SL == 8 || C::SL == 16, "slice layout");
      const int u = wm * 2 + g;
      const int ibase = (u / TPU) * 32 + 8 * (u % TPU) * (C::SL / 4);
#pragma unroll
      for (int s = 0; s < MW; ++s) {
        uint32_t w[C::SL / 4];
#pragma unroll
        for (int wi = 0; wi < C::SL / 4; ++wi) {
          uint32_t x = 0;
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float v = val[((4 * wi + e) * MW + s) * 2 + h];
              x |= code(v) << (4 * (4 * h + e));
              if constexpr (DBG) {
                if (c < A) args.dbg[row * C::K + c * B + ibase + s * C::MT * 32 + 8 * wi + 4 * h + e] = __fmul_rn(v, s_n);
              }
            }
          w[wi] = x;
        }
        if (c < A) {
          uint8_t* dst = qrow + (c * B + ibase + s * C::MT * 32) / 2;
          if constexpr (C::SL == 4) {
            *reinterpret_cast<uint32_t*>(dst) = w[0];
          } else if constexpr (C::SL == 8) {
            *reinterpret_cast<uint2*>(dst) = make_uint2(w[0], w[1]);
          } else {
            *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
          }
        }
      }
    }
    if constexpr (STAGE) {
      if (next < rows) store_stage();  // every wave is past its last read of lds_row
    }
    // the next row rewrites lds_red (and lds_row / lds_xch): all waves must be done with them
    __syncthreads();
  }
}

// ---------------------------------------------------------------- row-pair kernel (b = 64)
// Rows of K = A * 64 (H_A (x) S_64).  Two waves share a row; a workgroup of 8 waves (two
// per SIMD) works on 4 rows at a time, one LDS slot per row, one workgroup per CU.
//   * slot: the row as APAD lines of 128 bytes (64 fp16, one i_a each), lines A..APAD-1
//     zero; on odd lines the two 64-byte halves are swapped, so that the 8 lines one
//     transposing read touches fall evenly on the two bank halves;
//   * A fragments (8 consecutive i_a of one column i_b) come from two ds_read_b64_tr_b16:
//     within each 16-lane group the instruction hands lane i element e = word i % 4 of the
//     8-byte segment addressed by lane 4e + i / 4, so lane s addresses line
//     kbase + 4t + s / 4, columns 4 (s % 4) .. +3 of its half (t = 0, 1: k 0-3 and 4-7);
//   * the B fragments of H_A (fp16 +-1) sit in LDS, built once per workgroup; each wave of
//     the pair takes NT/2 of the MFMA N tiles (the columns j_a), so neither wave needs the
//     other's values;
//   * the next rows are loaded with 16-byte loads into registers while the current rows
//     are transformed, and written to their slots once both waves of a row have read it;
//   * Sylvester stages over i_b in registers, plus one lane-half stage by
//     v_permlane32_swap; per-row min/max (the two waves of a row meet in LDS); codes use
//     one fma per value and v_cvt_pk_u8_f32 (round half to even), which can move a code
//     by one only on a rounding boundary;
//   * the two waves of a row synchronise with each other only (progress counters in LDS),
//     never with the other rows' waves, so each pair starts as soon as its own row is in.
template <int A, int APAD, int NT>
struct Pair {
  static constexpr int B = 64;
  static constexpr int K = A * B;
  static constexpr int KS = APAD / 16;        // k-steps of the dense stage over i_a
  static constexpr int MT = 2;                // M tiles (32 i_b each)
  static constexpr int NTW = NT / 2;          // N tiles per wave
  static constexpr int ROWS = 4;              // rows per workgroup iteration
  static constexpr int THREADS = 64 * 2 * ROWS;
  static constexpr int CHUNKS = K / 8;                   // 16-byte chunks of a row
  static constexpr int PF = (CHUNKS + 127) / 128;        // chunks per lane of the wave pair
  static constexpr int HFRAG = KS * NT * 64;             // 16-byte B fragments
  static constexpr int SLOT = APAD * 128;                // bytes of one staged row
  static constexpr int ZERO_CHUNKS = (APAD - A) * 8;     // zero padding lines of a slot
  static constexpr int RED = 2 * ROWS * 2 * 2;           // floats: [parity][row][wave][min,max]
  static constexpr int FLAGS = 2 * ROWS * 2;             // ints: [kind][row][wave] progress counters
  static constexpr int LDS = HFRAG * 16 + ROWS * SLOT + RED * 4 + FLAGS * 4;
  static_assert(NT % 2 == 0 && NT * 32 >= A, "N tiles");
  static_assert(APAD % 16 == 0 && APAD >= A && A % 4 == 0, "padding");
  static_assert(ZERO_CHUNKS <= 128, "one zero chunk per thread of a wave pair");
};

typedef short v4s __attribute__((ext_vector_type(4)));

// Progress counter of wave `me` of a row pair: published after the wave's LDS writes, and
// awaited (counter of the partner wave >= target) before reading what the partner wrote.
__device__ __forceinline__ void pair_publish(int* flag, int value) {
  __hip_atomic_store(flag, value, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void pair_wait(const int* flag, int target) {
  while (__hip_atomic_load(flag, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < target)
    __builtin_amdgcn_s_sleep(1);
}

template <int A, int APAD, int NT, bool DBG, int BITS, bool VAR>
__global__ void __launch_bounds__(512, 2)
had_quant_pair(RotQuantArgs args) {
  using C = Pair<A, APAD, NT>;
  constexpr int B = C::B;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  v8h* hf = reinterpret_cast<v8h*>(smem);
  unsigned char* slots = smem + C::HFRAG * 16;
  float* red = reinterpret_cast<float*>(smem + C::HFRAG * 16 + C::ROWS * C::SLOT);
  int* flags = reinterpret_cast<int*>(smem + C::HFRAG * 16 + C::ROWS * C::SLOT + C::RED * 4);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int p = wave >> 1;  // row slot
  const int h = wave & 1;   // which half of the N tiles
  const int g = lane >> 5;
  const int c = lane & 31;
  const int pl = h * 64 + lane;  // lane index within the wave pair (row staging)
  const int64_t rows = args.rows;
  const int64_t nsets = (rows + C::ROWS - 1) / C::ROWS;
  int64_t rs = blockIdx.x;
  if (rs >= nsets) return;  // uniform over the workgroup

  // ---- row staging: the wave pair loads chunk pl + 128 j of its row (16 bytes each)
  unsigned char* slot = slots + p * C::SLOT;
  v4u pf[C::PF];
  auto load_row = [&](int64_t r) {
    const v4u* xr = reinterpret_cast<const v4u*>(args.x + r * args.ldx);
#pragma unroll
    for (int j = 0; j < C::PF; ++j) {
      const int i = pl + 128 * j;
      pf[j] = xr[i < C::CHUNKS ? i : C::CHUNKS - 1];
    }
  };
  auto store_row = [&]() {
    if constexpr (VAR) {
      if (args.signs) {  // S flips element signs as the row goes to its slot
        const uint2* sg = reinterpret_cast<const uint2*>(args.signs);
        uint2 sv[C::PF];
#pragma unroll
        for (int j = 0; j < C::PF; ++j) {
          const int i = pl + 128 * j;
          sv[j] = sg[i < C::CHUNKS ? i : C::CHUNKS - 1];
        }
#pragma unroll
        for (int j = 0; j < C::PF; ++j) pf[j] ^= sign_mask(sv[j]);
      }
    }
#pragma unroll
    for (int j = 0; j < C::PF; ++j) {
      const int i = pl + 128 * j;  // line i / 8, chunk i % 8; odd lines swap their halves
      if (i < C::CHUNKS) reinterpret_cast<v4u*>(slot)[i ^ ((i & 8) >> 1)] = pf[j];
    }
  };
  // ---- H_A (int8 [A][A]) with coalesced 16-byte loads, issued before the first rows so
  //      that waiting for it does not wait for them; staged as bytes in the (still empty)
  //      slot area, from which the MFMA B fragments are built while the rows are in flight
  constexpr int HCH = (A * A + 15) / 16;                  // 16-byte chunks of H
  constexpr int HPT = (HCH + C::THREADS - 1) / C::THREADS;
  static_assert(HCH * 16 <= C::ROWS * C::SLOT, "H staging fits the slots");
  v4u hv[HPT];
#pragma unroll
  for (int j = 0; j < HPT; ++j) {
    const int i = threadIdx.x + j * C::THREADS;
    if (i < HCH) {
      if (i * 16 + 16 <= A * A) {
        hv[j] = reinterpret_cast<const v4u*>(args.H)[i];
      } else {  // the tail chunk, byte by byte
        uint32_t w[4] = {0u, 0u, 0u, 0u};
        for (int b = 0; i * 16 + b < A * A; ++b)
          w[b >> 2] |= static_cast<uint32_t>(static_cast<uint8_t>(args.H[i * 16 + b])) << (8 * (b & 3));
        hv[j] = v4u{w[0], w[1], w[2], w[3]};
      }
    }
  }
  {  // the first rows are in flight while D is built
    const int64_t r0 = rs * C::ROWS + p;
    load_row(r0 < rows ? r0 : rows - 1);
  }
#pragma unroll
  for (int j = 0; j < HPT; ++j) {
    const int i = threadIdx.x + j * C::THREADS;
    if (i < HCH) reinterpret_cast<v4u*>(slots)[i] = hv[j];
  }
  if (threadIdx.x < C::FLAGS) flags[threadIdx.x] = 0;
  __syncthreads();

  // ---- H_A as MFMA B fragments: hf[(ks*NT + nt)*64 + l][e] = H[k][n] with k = ks*16 +
  //      8*(l/32) + e and n = nt*32 + l%32; zero where k or n >= A.  A thread owns one column
  //      (nt, l) of the staged bytes.
  {
    const int8_t* hs = reinterpret_cast<const int8_t*>(slots);
    for (int i = threadIdx.x; i < NT * 64; i += C::THREADS) {
      const int l = i & 63;
      const int nt = i >> 6;
      const int ja = nt * 32 + (l & 31);
      const int g8 = 8 * (l >> 5);
      const int8_t* hcol = hs + (ja < A ? ja : A - 1);
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        v8h f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int ia = ks * 16 + g8 + e;
          const float hv1 = static_cast<float>(hcol[(ia < A ? ia : A - 1) * A]);
          f[e] = (ia < A && ja < A) ? static_cast<_Float16>(hv1) : static_cast<_Float16>(0.0f);
        }
        hf[(ks * NT + nt) * 64 + l] = f;
      }
    }
  }
  __syncthreads();  // the staged bytes are no longer read: the slots take the rows
  if (pl < C::ZERO_CHUNKS)  // the pair's padding lines i_a >= A: zero, never rewritten
    reinterpret_cast<v4u*>(slot)[A * 8 + pl] = v4u{0u, 0u, 0u, 0u};
  // flags[k*2*ROWS + p*2 + h]: k = 0: min/max of iteration it published (it + 1);
  //                            k = 1: rows of iteration it stored to the slot (it + 1)
  int* const mine0 = flags + p * 2 + h;
  int* const mine1 = flags + 2 * C::ROWS + p * 2 + h;
  const int* const other0 = flags + p * 2 + (h ^ 1);
  const int* const other1 = flags + 2 * C::ROWS + p * 2 + (h ^ 1);
  // each pair starts as soon as its own first row is in its slot (counter value 1 before
  // iteration 0; later iterations publish it + 1 for the rows of iteration it + 1)
  store_row();
  if (lane == 0) pair_publish(mine1, 1);
  pair_wait(other1, 1);

  // transposing reads of A fragments: lane (group G = lane/16, s = lane%16) addresses line
  // 8*(G/2) + 4t + s/4 (+ 16 ks) and columns 32*mt + 16*(G%2) + 4*(s%4), whose half is
  // swapped when the line is odd (s/4 odd)
  const int tg = lane >> 4, ts = lane & 15;
  const int tq = ts >> 2;
  uint32_t tbase[C::MT];
#pragma unroll
  for (int mt = 0; mt < C::MT; ++mt)
    tbase[mt] = static_cast<uint32_t>(p * C::SLOT + (8 * (tg >> 1) + tq) * 128 +
                                      ((32 * (mt ^ (tq & 1))) + 16 * (tg & 1) + 4 * (ts & 3)) * 2);
  auto frag = [&](int mt, int ks) {
    const unsigned char* a0 = slots + tbase[mt] + ks * 16 * 128;
    const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        reinterpret_cast<__attribute__((address_space(3))) v4s*>(reinterpret_cast<uintptr_t>(a0)));
    const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        reinterpret_cast<__attribute__((address_space(3))) v4s*>(reinterpret_cast<uintptr_t>(a0 + 4 * 128)));
    return __builtin_bit_cast(v8h, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };

  const float s_n = args.inv_sqrt_n;
  for (int it = 0; rs < nsets; ++it, rs += gridDim.x) {
    const int64_t row = rs * C::ROWS + p;
    const bool valid = row < rows;
    const bool more = rs + gridDim.x < nsets;
    if (more) {  // next rows: in flight during this iteration
      const int64_t nr = (rs + gridDim.x) * C::ROWS + p;
      load_row(nr < rows ? nr : rows - 1);
    }

    // ---- dense stage: acc[mt][nt] = X2^T H for i_b tile mt, H column tile h*NTW + nt;
    //      both M tiles' fragments read a k-step ahead
    v16f acc[C::MT][C::NTW];
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < C::NTW; ++nt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mt][nt][r] = 0.0f;
    {
      // A and B fragments of k-step ks + 1 are read while the MFMAs of k-step ks run
      v8h a0[C::MT], a1[C::MT], b0[C::NTW], b1[C::NTW];
      const v8h* hb = hf + h * C::NTW * 64 + lane;
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt) a0[mt] = frag(mt, 0);
#pragma unroll
      for (int nt = 0; nt < C::NTW; ++nt) b0[nt] = hb[nt * 64];
      static_for<C::KS>([&](auto kc) {
        constexpr int ks = decltype(kc)::value;
        v8h(&cur)[C::MT] = (ks & 1) ? a1 : a0;
        v8h(&nxt)[C::MT] = (ks & 1) ? a0 : a1;
        v8h(&bcur)[C::NTW] = (ks & 1) ? b1 : b0;
        v8h(&bnxt)[C::NTW] = (ks & 1) ? b0 : b1;
        if constexpr (ks + 1 < C::KS) {
#pragma unroll
          for (int mt = 0; mt < C::MT; ++mt) nxt[mt] = frag(mt, ks + 1);
#pragma unroll
          for (int nt = 0; nt < C::NTW; ++nt) bnxt[nt] = hb[((ks + 1) * NT + nt) * 64];
        }
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < C::NTW; ++nt)
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(cur[mt], bcur[nt], acc[mt][nt], 0, 0, 0);
      });
    }

    // ---- Sylvester stages over i_b: register bits 0, 1, 3, 4; M tile bit 5; lane half bit 2
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < C::NTW; ++nt)
#pragma unroll
        for (int rb = 1; rb < 16; rb <<= 1)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if ((r & rb) == 0) {
              float lo = acc[mt][nt][r], hi = acc[mt][nt][r + rb];
              bfly(lo, hi);
              acc[mt][nt][r] = lo;
              acc[mt][nt][r + rb] = hi;
            }
#pragma unroll
    for (int nt = 0; nt < C::NTW; ++nt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float lo = acc[0][nt][r], hi = acc[1][nt][r];
        bfly(lo, hi);
        acc[0][nt][r] = lo;
        acc[1][nt][r] = hi;
      }
    // lane-half stage (i_b bit 2): v_permlane32_swap of registers r and r + 8 (r < 8) puts
    // both bit-2 partners of register r (lanes 0-31) or r + 8 (lanes 32-63) in one lane;
    // the butterfly then leaves lane (c, g) holding i_b = mt*32 + 16g + j in acc[mt][nt][j],
    // j = 8q + 4*bit2 + e, sixteen consecutive positions
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < C::NTW; ++nt) {
        float o[16];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[mt][nt][r]),
                                                           __float_as_uint(acc[mt][nt][r + 8]), false, false);
          const float x0 = __uint_as_float(sw[0]);  // bit 2 clear
          const float x1 = __uint_as_float(sw[1]);  // bit 2 set
          const int j = 8 * (r >> 2) + (r & 3);
          o[j] = __fadd_rn(x0, x1);
          o[j + 4] = __fsub_rn(x0, x1);
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[mt][nt][j] = o[j];
      }

    // ---- per-row min/max over real columns (a lane's columns past A hold zeros: merged
    //      per tile under one condition); the two waves of the row meet in LDS
    float mn = INFINITY, mx = -INFINITY;
#pragma unroll
    for (int nt = 0; nt < C::NTW; ++nt) {
      float tmn = acc[0][nt][0], tmx = acc[0][nt][0];
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          tmn = fminf(tmn, acc[mt][nt][r]);
          tmx = fmaxf(tmx, acc[mt][nt][r]);
        }
      if ((h * C::NTW + nt) * 32 + 32 <= A || (h * C::NTW + nt) * 32 + c < A) {
        mn = fminf(mn, tmn);
        mx = fmaxf(mx, tmx);
      }
    }
    mn = wave_min(mn);
    mx = wave_max(mx);
    // the two waves of the row meet: parity buffers, so a wave can be one iteration ahead
    float* rd = red + (it & 1) * (C::ROWS * 4);
    if (lane == 0) {
      rd[(p * 2 + h) * 2] = mn;
      rd[(p * 2 + h) * 2 + 1] = mx;
      pair_publish(mine0, it + 1);
    }
    pair_wait(other0, it + 1);  // also: the partner is done reading the slot
    mn = fminf(rd[p * 4], rd[p * 4 + 2]);
    mx = fmaxf(rd[p * 4 + 1], rd[p * 4 + 3]);
    if (more) {
      store_row();
      if (lane == 0) pair_publish(mine1, it + 2);
    }
    if constexpr (VAR) {  // clipped range [r min, r max]
      mn = __fmul_rn(mn, args.clip);
      mx = __fmul_rn(mx, args.clip);
    }

    // eq. 1 in the unscaled domain; reported alpha, beta carry the 1/sqrt(K) scale
    const float r_u = __fsub_rn(mx, mn);
    const float a_u = __fdiv_rn(r_u, BITS == 8 ? 255.0f : 15.0f);
    const bool cst = __fmul_rn(a_u, s_n) < kMinNormal;
    const float inv_u = cst ? 0.0f : __fdiv_rn(1.0f, a_u);
    const float nb = -__fmul_rn(mn, inv_u);
    if (valid && h == 0 && lane == 0) {
      args.alpha[row] = cst ? 1.0f : __fmul_rn(a_u, s_n);
      args.beta[row] = __fmul_rn(mn, s_n);
    }

    // ---- codes: lane (c, g) holds i_b = mt*32 + 16g + j (j = 0..15) of column j_a: bytes
    // via v_cvt_pk_u8_f32 (even j in ev, odd j in od), ev | od << 4 is then four
    // nibble-packed bytes; 8-byte store at output position j_a*64 + mt*32 + 16g.
    uint8_t* qrow = args.q + row * (C::K * BITS / 8);
#pragma unroll
    for (int nt = 0; nt < C::NTW; ++nt) {
      const int ja = (h * C::NTW + nt) * 32 + c;
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt) {
        const int pos = ja * B + mt * 32 + 16 * g;
        if constexpr (BITS == 8) {  // one code per byte: 16-byte store
          uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
          for (int j = 0; j < 16; ++j) w[j >> 2] = __builtin_amdgcn_cvt_pk_u8_f32(code_arg<VAR, BITS>(__fmaf_rn(acc[mt][nt][j], inv_u, nb)), j & 3, w[j >> 2]);
          if (valid && ja < A) *reinterpret_cast<uint4*>(qrow + pos) = make_uint4(w[0], w[1], w[2], w[3]);
        } else {
          uint32_t w[2];
#pragma unroll
          for (int hw = 0; hw < 2; ++hw) {
            uint32_t ev = 0, od = 0;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
              ev = __builtin_amdgcn_cvt_pk_u8_f32(code_arg<VAR, BITS>(__fmaf_rn(acc[mt][nt][8 * hw + 2 * s], inv_u, nb)), s, ev);
              od = __builtin_amdgcn_cvt_pk_u8_f32(code_arg<VAR, BITS>(__fmaf_rn(acc[mt][nt][8 * hw + 2 * s + 1], inv_u, nb)), s, od);
            }
            w[hw] = ev | (od << 4);
          }
          if (valid && ja < A) *reinterpret_cast<uint2*>(qrow + pos / 2) = make_uint2(w[0], w[1]);
        }
        if constexpr (DBG) {
          if (valid && ja < A) {
#pragma unroll
            for (int j = 0; j < 16; ++j) args.dbg[row * C::K + pos + j] = __fmul_rn(acc[mt][nt][j], s_n);
          }
        }
      }
    }
    if (more) pair_wait(other1, it + 2);  // the slot holds the next row, both halves
  }
}

// ---------------------------------------------------------------- line kernel
// Rows of K = A * F * 64 rotated by (H_A (x) S_{64F}) / sqrt(K).  The Sylvester factor
// splits as S_{64F} = S_F (x) S_64 (the left factor on the high index bits), so with the
// row viewed as AD = A*F lines of 64 fp16 (line L = i_a*F + i_b/64, column i_b % 64) the
// rotation is D (x) S_64 with D = H_A (x) S_F of order AD acting on the line index.  F = 8
// turns H_28 (x) S_512 into a 224-line dense stage with no padding (H_28 (x) S_1024: F = 16,
// 448 lines), and the butterflies that remain (S_64) stay inside a line.
//   * one workgroup of NT waves owns one row at a time; wave w computes the 32 output lines
//     n = 32w .. 32w + 31 (one MFMA N tile) over all 64 columns (two M tiles), so every
//     butterfly of the S_64 stage is inside the wave and the waves meet only for the row's
//     min/max;
//   * the B fragments (columns of D) stay in registers for the whole kernel: F being a
//     multiple of 8, a fragment (8 consecutive k) lies in one entry of H_A, so a lane keeps
//     one fp16 +-1 pattern of S_F and applies the H_A sign per k-step by flipping fp16 sign
//     bits (the fragments themselves, 4 VGPRs per k-step, would not fit beside the row);
//   * the row sits in LDS as APAD lines of 128 bytes (lines AD.. zero, odd lines with their
//     64-byte halves swapped) and A fragments come from transposing reads, as in the
//     row-pair kernel; the next row is loaded into registers while this one is transformed;
//   * several workgroups share a CU, so one's loads, MFMAs and VALU work overlap another's.
template <int A, int F, int NT>
struct Lines {
  static constexpr int AD = A * F;                    // lines of a row
  static constexpr int KS = (AD + 15) / 16;           // k-steps of the dense stage
  static constexpr int APAD = KS * 16;                // staged lines
  static constexpr int K = AD * 64;
  static constexpr int THREADS = 64 * NT;
  static constexpr int CHUNKS = K / 8;                // 16-byte chunks of a row
  static constexpr int PF = (CHUNKS + THREADS - 1) / THREADS;
  static constexpr int SLOT = APAD * 128;
  static constexpr int ZERO_CHUNKS = (APAD - AD) * 8;
  static constexpr int HCH = (A * A + 15) / 16;       // 16-byte chunks of H_A
  static constexpr int HPT = (HCH + THREADS - 1) / THREADS;
  static constexpr int STAGE = SLOT > HCH * 16 ? SLOT : HCH * 16;  // row slot, or H at the start
  static constexpr int LDS = STAGE + 2 * NT * 4;      // + per-wave min/max
  static_assert(F == 8 || F == 16, "a fragment in one H_A entry, one S_F pattern for all k-steps");
  static_assert(NT * 32 >= AD && (NT - 1) * 32 < AD, "one N tile per wave, none empty");
  static_assert(ZERO_CHUNKS <= THREADS, "padding lines zeroed in one pass");
  static_assert(KS <= 32, "k-step sign bits");
};

template <int A, int F, int NT, bool DBG, int BITS, bool VAR>
__global__ void __launch_bounds__(64 * NT, DBG ? 2 : 4)  // 4 waves per SIMD: 128 VGPRs
had_quant_lines(RotQuantArgs args) {
  using C = Lines<A, F, NT>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* slot = smem;
  float* red = reinterpret_cast<float*>(smem + C::STAGE);
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int g = lane >> 5;
  const int c = lane & 31;
  const int n = 32 * w + c;  // output line (column of D) of this lane
  const int64_t rows = args.rows;
  int64_t row = blockIdx.x;
  if (row >= rows) return;  // uniform over the workgroup

  // ---- row staging: thread t loads chunks t + THREADS * j (clamped in the row; the
  //      duplicates are not stored)
  v4u pf[C::PF];
  auto load_row = [&](int64_t r) {
    const v4u* xr = reinterpret_cast<const v4u*>(args.x + r * args.ldx);
#pragma unroll
    for (int j = 0; j < C::PF; ++j) {
      const int i = threadIdx.x + C::THREADS * j;
      pf[j] = xr[i < C::CHUNKS ? i : C::CHUNKS - 1];
    }
  };
  auto store_row = [&]() {
    if constexpr (VAR) {
      if (args.signs) {  // S flips element signs as the row goes to the slot
        const uint2* sg = reinterpret_cast<const uint2*>(args.signs);
        uint2 sv[C::PF];
#pragma unroll
        for (int j = 0; j < C::PF; ++j) {
          const int i = threadIdx.x + C::THREADS * j;
          sv[j] = sg[i < C::CHUNKS ? i : C::CHUNKS - 1];
        }
#pragma unroll
        for (int j = 0; j < C::PF; ++j) pf[j] ^= sign_mask(sv[j]);
      }
    }
#pragma unroll
    for (int j = 0; j < C::PF; ++j) {
      const int i = threadIdx.x + C::THREADS * j;  // line i / 8, chunk i % 8
      if (i < C::CHUNKS) reinterpret_cast<v4u*>(slot)[i ^ ((i & 8) >> 1)] = pf[j];
    }
  };
  // H_A (int8 [A][A]) with coalesced 16-byte loads, staged as bytes in the slot (the rows
  // go there once the fragments are built); the first row is requested first
  load_row(row);
  {
    v4u hv[C::HPT];
#pragma unroll
    for (int j = 0; j < C::HPT; ++j) {
      const int i = threadIdx.x + j * C::THREADS;
      if (i < C::HCH) {
        if (i * 16 + 16 <= A * A) {
          hv[j] = reinterpret_cast<const v4u*>(args.H)[i];
        } else {  // the tail chunk, byte by byte
          uint32_t wd[4] = {0u, 0u, 0u, 0u};
          for (int b = 0; i * 16 + b < A * A; ++b)
            wd[b >> 2] |= static_cast<uint32_t>(static_cast<uint8_t>(args.H[i * 16 + b])) << (8 * (b & 3));
          hv[j] = v4u{wd[0], wd[1], wd[2], wd[3]};
        }
      }
    }
#pragma unroll
    for (int j = 0; j < C::HPT; ++j) {
      const int i = threadIdx.x + j * C::THREADS;
      if (i < C::HCH) reinterpret_cast<v4u*>(slot)[i] = hv[j];
    }
  }
  __syncthreads();
  const int8_t* hs = reinterpret_cast<const int8_t*>(slot);

  // ---- B fragments: B[k][n] = D[k][n] for k = 16 ks + 8 g + e; zero where k or n >= AD
  // k = (16 ks + 8 g) + e: the fragment lies in H_A entry [(16 ks + 8 g) / F][n / F] and
  // in S_F rows (8 g) % F + e, column n % F (the reads use clamped indices and are
  // unconditional, so that they are all in flight at once)
  v8h bf;
  uint32_t sgn = 0;  // bit ks set when the k-step's H_A entry is -1
  {
    const int nt = n % F;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int kt = (8 * g) % F + e;
      bf[e] = (n < C::AD) ? static_cast<_Float16>((__popc(kt & nt) & 1) ? -1.0f : 1.0f)
                          : static_cast<_Float16>(0.0f);
    }
    const int na = n < C::AD ? n / F : A - 1;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      const int ka = (16 * ks + 8 * g) / F;
      const int8_t h = hs[(ka < A ? ka : A - 1) * A + na];
      if (ka < A && n < C::AD && h < 0) sgn |= 1u << ks;
    }
  }
  __syncthreads();  // the staged H is no longer read: the slot takes the rows
  if (threadIdx.x < C::ZERO_CHUNKS)  // padding lines: zero, never rewritten
    reinterpret_cast<v4u*>(slot)[C::AD * 8 + threadIdx.x] = v4u{0u, 0u, 0u, 0u};
  store_row();
  __syncthreads();

  // transposing reads of A fragments (see the row-pair kernel): lane (G = lane/16,
  // s = lane%16) addresses line 8*(G/2) + 4t + s/4 (+ 16 ks), columns 32*mt + 16*(G%2) +
  // 4*(s%4), half-swapped on odd lines
  const int tg = lane >> 4, ts = lane & 15;
  const int tq = ts >> 2;
  uint32_t tbase[2];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
    tbase[mt] = static_cast<uint32_t>((8 * (tg >> 1) + tq) * 128 +
                                      ((32 * (mt ^ (tq & 1))) + 16 * (tg & 1) + 4 * (ts & 3)) * 2);
  auto frag = [&](int mt, int ks) {
    const unsigned char* a0 = slot + tbase[mt] + ks * 16 * 128;
    const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        reinterpret_cast<__attribute__((address_space(3))) v4s*>(reinterpret_cast<uintptr_t>(a0)));
    const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        reinterpret_cast<__attribute__((address_space(3))) v4s*>(reinterpret_cast<uintptr_t>(a0 + 4 * 128)));
    return __builtin_bit_cast(v8h, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  auto bfrag = [&](int ks) {
    const uint32_t m = ((sgn >> ks) & 1u) ? 0x80008000u : 0u;
    v4u b = __builtin_bit_cast(v4u, bf);
    b ^= v4u{m, m, m, m};
    return __builtin_bit_cast(v8h, b);
  };

  const float s_n = args.inv_sqrt_n;
  const bool real = n < C::AD;
  for (;;) {
    const int64_t next = row + gridDim.x;
    const bool more = next < rows;
    if (more) load_row(next);  // in flight during this row
    // keeps the sign flips inside the loop (hoisted out of it, the flipped fragments would
    // take 4 VGPRs per k-step)
    asm volatile("" : "+v"(sgn));

    // ---- dense stage: acc[mt] = (X lines)^T D for columns 32 mt .. 32 mt + 31
    v16f acc[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mt][r] = 0.0f;
    {
      v8h a0[2], a1[2];
      a0[0] = frag(0, 0);
      a0[1] = frag(1, 0);
      static_for<C::KS>([&](auto kc) {
        constexpr int ks = decltype(kc)::value;
        v8h(&cur)[2] = (ks & 1) ? a1 : a0;
        v8h(&nxt)[2] = (ks & 1) ? a0 : a1;
        if constexpr (ks + 1 < C::KS) {
          nxt[0] = frag(0, ks + 1);
          nxt[1] = frag(1, ks + 1);
        }
        const v8h b = bfrag(ks);
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(cur[0], b, acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(cur[1], b, acc[1], 0, 0, 0);
      });
    }

    // ---- S_64 over the column: register bits 0, 1, 3, 4; M tile bit 5; lane half bit 2
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int rb = 1; rb < 16; rb <<= 1)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if ((r & rb) == 0) {
            float lo = acc[mt][r], hi = acc[mt][r + rb];
            bfly(lo, hi);
            acc[mt][r] = lo;
            acc[mt][r + rb] = hi;
          }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float lo = acc[0][r], hi = acc[1][r];
      bfly(lo, hi);
      acc[0][r] = lo;
      acc[1][r] = hi;
    }
    // after the swap and butterfly lane (c, g) holds column 32 mt + 16 g + j in acc[mt][j]
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      float o[16];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[mt][r]),
                                                         __float_as_uint(acc[mt][r + 8]), false, false);
        const float x0 = __uint_as_float(sw[0]);
        const float x1 = __uint_as_float(sw[1]);
        const int j = 8 * (r >> 2) + (r & 3);
        o[j] = __fadd_rn(x0, x1);
        o[j + 4] = __fsub_rn(x0, x1);
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[mt][j] = o[j];
    }

    // ---- row min/max over real lines (padding lines hold zeros)
    float mn = acc[0][0], mx = acc[0][0];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        mn = fminf(mn, acc[mt][r]);
        mx = fmaxf(mx, acc[mt][r]);
      }
    if (!real) {
      mn = INFINITY;
      mx = -INFINITY;
    }
    mn = wave_min(mn);
    mx = wave_max(mx);
    if (lane == 0) {
      red[w] = mn;
      red[NT + w] = mx;
    }
    __syncthreads();  // every wave is past its dense stage: the slot may take the next row
    mn = red[0];
    mx = red[NT];
#pragma unroll
    for (int v = 1; v < NT; ++v) {
      mn = fminf(mn, red[v]);
      mx = fmaxf(mx, red[NT + v]);
    }
    if (more) store_row();
    if constexpr (VAR) {  // clipped range [r min, r max]
      mn = __fmul_rn(mn, args.clip);
      mx = __fmul_rn(mx, args.clip);
    }

    // eq. 1 in the unscaled domain; reported alpha, beta carry the 1/sqrt(K) scale
    const float r_u = __fsub_rn(mx, mn);
    const float a_u = __fdiv_rn(r_u, BITS == 8 ? 255.0f : 15.0f);
    const bool cst = __fmul_rn(a_u, s_n) < kMinNormal;
    const float inv_u = cst ? 0.0f : __fdiv_rn(1.0f, a_u);
    const float nb = -__fmul_rn(mn, inv_u);
    if (threadIdx.x == 0) {
      args.alpha[row] = cst ? 1.0f : __fmul_rn(a_u, s_n);
      args.beta[row] = __fmul_rn(mn, s_n);
    }

    // ---- codes of line n, columns 32 mt + 16 g .. + 15: 8-byte stores
    uint8_t* qrow = args.q + row * (C::K * BITS / 8);
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const int pos = n * 64 + mt * 32 + 16 * g;
      if constexpr (BITS == 8) {  // one code per byte: 16-byte store
        uint32_t wd[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int j = 0; j < 16; ++j) wd[j >> 2] = __builtin_amdgcn_cvt_pk_u8_f32(code_arg<VAR, BITS>(__fmaf_rn(acc[mt][j], inv_u, nb)), j & 3, wd[j >> 2]);
        if (real) *reinterpret_cast<uint4*>(qrow + pos) = make_uint4(wd[0], wd[1], wd[2], wd[3]);
      } else {
        uint32_t wd[2];
#pragma unroll
        for (int hw = 0; hw < 2; ++hw) {
          uint32_t ev = 0, od = 0;
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            ev = __builtin_amdgcn_cvt_pk_u8_f32(code_arg<VAR, BITS>(__fmaf_rn(acc[mt][8 * hw + 2 * s], inv_u, nb)), s, ev);
            od = __builtin_amdgcn_cvt_pk_u8_f32(code_arg<VAR, BITS>(__fmaf_rn(acc[mt][8 * hw + 2 * s + 1], inv_u, nb)), s, od);
          }
          wd[hw] = ev | (od << 4);
        }
        if (real) *reinterpret_cast<uint2*>(qrow + pos / 2) = make_uint2(wd[0], wd[1]);
      }
      if constexpr (DBG) {
        if (real) {
#pragma unroll
          for (int j = 0; j < 16; ++j) args.dbg[row * C::K + pos + j] = __fmul_rn(acc[mt][j], s_n);
        }
      }
    }
    __syncthreads();  // the slot holds the next row; the min/max slots are free again
    if (!more) break;
    row = next;
  }
}

// Compute units of the current device (the persistent grids' size); if the query fails,
// 256 (MI355X): the grid then only runs in fewer or more rounds.
int num_cus() {
  int n = 0;
  return device_cus(&n) == hipSuccess ? n : 256;
}

template <int A, int APAD, int NT, int B, int MW, int NW, bool STAGE, bool DBG>
hipError_t launch_kron_t(const RotQuantArgs& a, hipStream_t stream) {
  using C = Kron<A, APAD, NT, B, MW, NW, STAGE>;
  constexpr auto kern = had_quant_kron<A, APAD, NT, B, MW, NW, STAGE, DBG>;
  hipError_t e = set_max_lds<kern>(C::LDS);
  int per_cu = 1;
  if (e == hipSuccess) e = blocks_per_cu<kern>(C::THREADS, C::LDS, &per_cu);
  if (e != hipSuccess) return e;
  const int64_t cap = static_cast<int64_t>(num_cus()) * per_cu;
  const unsigned grid = static_cast<unsigned>(a.rows < cap ? a.rows : cap);
  return launch(kern, dim3(grid), dim3(C::THREADS), C::LDS, stream, a);
}

template <int A, int APAD, int NT, int B, int MW, int NW, bool STAGE>
hipError_t launch_kron(const RotQuantArgs& a, hipStream_t stream) {
  return a.dbg ? launch_kron_t<A, APAD, NT, B, MW, NW, STAGE, true>(a, stream)
               : launch_kron_t<A, APAD, NT, B, MW, NW, STAGE, false>(a, stream);
}

template <int A, int APAD, int NT, bool DBG, int BITS, bool VAR>
hipError_t launch_pair_t(const RotQuantArgs& a, hipStream_t stream) {
  using C = Pair<A, APAD, NT>;
  constexpr auto kern = had_quant_pair<A, APAD, NT, DBG, BITS, VAR>;
  const hipError_t init = set_max_lds<kern>(C::LDS);
  if (init != hipSuccess) return init;
  const int64_t sets = (a.rows + C::ROWS - 1) / C::ROWS;
  const int64_t cap = num_cus();
  const unsigned grid = static_cast<unsigned>(sets < cap ? sets : cap);
  return launch(kern, dim3(grid), dim3(C::THREADS), C::LDS, stream, a);
}

// Calls f(dbg, b8, var) with each flag as a std::bool_constant, so that one call site
// instantiates every combination of the kernels' compile-time switches.
template <typename Fn>
hipError_t with_flags(bool dbg, bool b8, bool var, Fn&& f) {
  using T = std::true_type;
  using N = std::false_type;
  if (dbg) {
    if (b8) return var ? f(T{}, T{}, T{}) : f(T{}, T{}, N{});
    return var ? f(T{}, N{}, T{}) : f(T{}, N{}, N{});
  }
  if (b8) return var ? f(N{}, T{}, T{}) : f(N{}, T{}, N{});
  return var ? f(N{}, N{}, T{}) : f(N{}, N{}, N{});
}

bool is_variant(const RotQuantArgs& a) { return a.clip != 1.0f || a.signs != nullptr; }

template <int A, int APAD, int NT>
hipError_t launch_pair(const RotQuantArgs& a, hipStream_t stream) {
  return with_flags(a.dbg != nullptr, a.bits == 8, is_variant(a), [&](auto dbg, auto b8, auto var) {
    return launch_pair_t<A, APAD, NT, decltype(dbg)::value, decltype(b8)::value ? 8 : 4, decltype(var)::value>(a, stream);
  });
}

template <int A, int F, int NT, bool DBG, int BITS, bool VAR>
hipError_t launch_lines_t(const RotQuantArgs& a, hipStream_t stream) {
  using C = Lines<A, F, NT>;
  constexpr auto kern = had_quant_lines<A, F, NT, DBG, BITS, VAR>;
  hipError_t e = set_max_lds<kern>(C::LDS);
  int per_cu = 1;
  if (e == hipSuccess) e = blocks_per_cu<kern>(C::THREADS, C::LDS, &per_cu);
  if (e != hipSuccess) return e;
  const int64_t cap = static_cast<int64_t>(num_cus()) * per_cu;
  const unsigned grid = static_cast<unsigned>(a.rows < cap ? a.rows : cap);
  return launch(kern, dim3(grid), dim3(C::THREADS), C::LDS, stream, a);
}

template <int A, int F, int NT>
hipError_t launch_lines(const RotQuantArgs& a, hipStream_t stream) {
  return with_flags(a.dbg != nullptr, a.bits == 8, is_variant(a), [&](auto dbg, auto b8, auto var) {
    return launch_lines_t<A, F, NT, decltype(dbg)::value, decltype(b8)::value ? 8 : 4, decltype(var)::value>(a, stream);
  });
}

}  // namespace

// Returns hipErrorNotSupported when no fast path covers the arguments.
hipError_t launch_had_quant_kron(const RotQuantArgs& a, hipStream_t stream) {
  if ((a.bits != 4 && a.bits != 8) || a.group != a.K || a.K != static_cast<int64_t>(a.a) * a.b || a.H == nullptr)
    return hipErrorNotSupported;
  // the pair and line kernels stage rows in 16-byte chunks (and write 4- or 8-bit codes,
  // with or without the clipping and sign variants; S is read 8 entries at a time); the
  // register-prefetch kernels write plain 4-bit codes only
  const bool pair_ok = (reinterpret_cast<uintptr_t>(a.x) & 15) == 0 && (a.ldx % 8) == 0 &&
                       (reinterpret_cast<uintptr_t>(a.H) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(a.signs) & 7) == 0;
  if (!pair_ok && (a.bits != 4 || is_variant(a))) return hipErrorNotSupported;
  if (a.a == 28 && a.b == 512) {
    if (pair_ok) return launch_lines<28, 8, 7>(a, stream);
    return launch_kron<28, 32, 1, 512, 4, 1, false>(a, stream);
  }
  if (a.a == 172 && a.b == 64) {
    if (pair_ok) return launch_pair<172, 176, 6>(a, stream);
    return launch_kron<172, 176, 6, 64, 1, 6, true>(a, stream);
  }
  if (a.a == 28 && a.b == 1024) {
    if (pair_ok) return launch_lines<28, 16, 14>(a, stream);
    return launch_kron<28, 32, 1, 1024, 8, 1, false>(a, stream);
  }
  return hipErrorNotSupported;
}

}  // namespace sq
