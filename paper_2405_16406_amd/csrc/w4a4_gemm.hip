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
// the dot product.  |16 acc| <= 16 * 15 * 7 * K < 2^31 for K < 1.2M.
//
// Main kernel (w4a4_gemm_ring): the packed operand tiles stream from global memory into
// an LDS ring by direct-to-LDS buffer loads, several stages ahead; each wave reads its
// fragments back with ds_read_b128, expands them with VALU and issues the MFMAs.  Tile
// shapes: 128 x 128 (4 waves of 64 x 64) for small M, 256 x 128 (4 waves of 128 x 64,
// two workgroups per CU) and 256 x 256 (8 waves of 128 x 64).
// Register-staged kernel (w4a4_gemm_tile): global -> registers -> LDS, double-buffered;
// used where 32-bit buffer offsets do not cover the operands.
// Decode sizes: w4a4_gemv (M <= 2: whole weight rows streamed through v_dot8_i32_i4),
// w4a4_gemm_stream (M <= 16, 8-bit activations M <= 8: weight and
// activation row segments copied into LDS, v_mfma_i32_16x16x64_i8) and w4a4_gemm_skinny
// (the remaining M <= 16 cases: weight rows straight into registers).
#include <utility>

#include "sq_device.h"
#include "sq_internal.h"

namespace sq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef unsigned v2u __attribute__((ext_vector_type(2)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));
typedef float v2f __attribute__((ext_vector_type(2)));

// The epilogue rounds twice, fp32 then fp16 (round to nearest even), in both of its paths.
// fp32_result pins a value as a rounded fp32 register so that the compiler cannot fuse the
// final fma with the fp16 conversion into one single-rounding v_fma_mix.  The asm is not
// volatile: it only hides the value, and the scheduler stays free to interleave the
// independent outputs (volatile asm statements keep their program order, which serialised
// the epilogue's long-latency exp and reciprocal steps).
__device__ __forceinline__ float fp32_result(float v) {
  asm("" : "+v"(v));
  return v;
}
// two fp32 -> two fp16 (round to nearest even), packed low | high << 16
__device__ __forceinline__ uint32_t f2h2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v2f{lo, hi}, v2h));
}

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

// Calls f(std::integral_constant<int, I>) for I = 0 .. N-1: indices into register arrays
// stay compile-time constants even where the unroller would give up.
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Epilogue of one 32 x 32 block held by a wave: lane holds C[8*(r/4) + 4*(lane/32) + r%4][lane%32].
__device__ __forceinline__ void store_block(const GemmArgs& g, const v16i& acc, int64_t m_base, int64_t n,
                                            int lane) {
  if (n >= g.N) return;
  const float sn = g.wa[n];
  const float rsn = static_cast<float>(g.rs[n]);
  const float bn = g.bias ? h2f(g.bias[n]) : 0.0f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int64_t m = m_base + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    if (m >= g.M) continue;
    const int a = acc[r] >> 4;
    if (g.dbg_acc) g.dbg_acc[m * g.N + n] = a;
    const float t = __fadd_rn(__fmul_rn(g.xa[m], static_cast<float>(a)), __fmul_rn(g.xb[m], rsn));
    float yv = __fmul_rn(sn, t);
    if (g.bias) yv = __fadd_rn(yv, bn);
    g.y[m * g.ldy + n] = f2h(yv);
  }
}

// Tile order.  Consecutive workgroup ids go to different XCDs (round robin over 8), so each
// XCD is given a contiguous range of tile ids; within it the tile walks M fastest, so the
// CUs of one XCD share weight (B) tiles in their L2 and each weight tile is read from HBM
// about once.  Grid: x = tiles along N, y = tiles along M.
__device__ __forceinline__ void tile_origin(int bm, int bn, int64_t& m0, int64_t& n0) {
  const int tiles_m = gridDim.y;
  const int total = gridDim.x * gridDim.y;
  const int bid = blockIdx.y * gridDim.x + blockIdx.x;
  const int q8 = total / 8, r8 = total % 8;
  const int xcd = bid % 8, idx = bid / 8;
  const int tile = xcd < r8 ? xcd * (q8 + 1) + idx : r8 * (q8 + 1) + (xcd - r8) * q8 + idx;
  m0 = static_cast<int64_t>(tile % tiles_m) * bm;
  n0 = static_cast<int64_t>(tile / tiles_m) * bn;
}

// y = (alpha_m s_n) acc + beta_m (s_n rs_n) [+ bias_n] for the TM x TN blocks of one wave,
// whose top-left output is (mw, nw); one fma per output.  Neighbouring columns sit in
// neighbouring lanes; even lanes store both as one 32-bit word when the output rows are
// 4-byte aligned.  One 32 x 32 block row at a time (sched_barrier keeps the scheduler from
// hoisting every block's accumulators at once).
template <int TM, int TN>
__device__ __forceinline__ void tile_epilogue(const GemmArgs& g, const v16i (&acc)[TM][TN], int64_t mw, int64_t nw,
                                              int lane) {
  const bool pair = ((g.ldy & 1) == 0) && ((reinterpret_cast<uintptr_t>(g.y) & 3) == 0) && (g.dbg_acc == nullptr);
  const int c = lane & 31;
  float csn[TN], cwr[TN], cbn[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int64_t n = nw + j * 32 + c;
    const int64_t nc = n < g.N ? n : g.N - 1;
    csn[j] = g.wa[nc];
    cwr[j] = __fmul_rn(csn[j], static_cast<float>(g.rs[nc]));
    cbn[j] = g.bias ? h2f(g.bias[nc]) : 0.0f;
  }
  static_for<TM>([&](auto ic) {
    constexpr int i = decltype(ic)::value;
    __builtin_amdgcn_sched_barrier(0);
    const int64_t mb = mw + i * 32 + 4 * (lane >> 5);
    float ra_[16], rb_[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t m = mb + 8 * (r >> 2) + (r & 3);
      const int64_t mc = m < g.M ? m : g.M - 1;
      ra_[r] = g.xa[mc];
      rb_[r] = g.xb[mc];
    }
    static_for<TN>([&](auto jc) {
      constexpr int j = decltype(jc)::value;
      const int64_t n = nw + j * 32 + c;
      const bool nok = n < g.N;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = mb + 8 * (r >> 2) + (r & 3);
        const bool mok = m < g.M;
        const int a = acc[i][j][r] >> 4;
        float yv = __fmaf_rn(__fmul_rn(ra_[r], csn[j]), static_cast<float>(a), __fmul_rn(rb_[r], cwr[j]));
        if (g.bias) yv = __fadd_rn(yv, cbn[j]);
        const uint32_t h = f2h(yv);
        if (pair) {
          // quad_perm [1,0,3,2]: each lane receives its neighbour's value
          const uint32_t other = static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(h), 0xB1, 0xF, 0xF, false));
          if ((c & 1) == 0 && mok && nok) {
            if (n + 1 < g.N)
              *reinterpret_cast<uint32_t*>(g.y + m * g.ldy + n) = h | (other << 16);
            else
              g.y[m * g.ldy + n] = static_cast<uint16_t>(h);
          }
        } else if (mok && nok) {
          if (g.dbg_acc) g.dbg_acc[m * g.N + n] = a;
          g.y[m * g.ldy + n] = static_cast<uint16_t>(h);
        }
      }
    });
  });
}

// Epilogue of the ring kernel.  Its MFMAs take the weights as the A operand, so each 32 x 32
// block is D[n][m]: lane (c, h) = (lane % 32, lane / 32) holds row m = mb + c and columns
// n = nb + 8q + 4h + e in registers r = 4q + e, i.e. four consecutive outputs of one row per
// q, written with one 8-byte store.  The accumulators hold 16 * acc (weights expanded as
// 16 * code), so alpha_m / 16 is applied:
//   y = fma(alpha_m/16, s_n * acc16, fma(beta_m, s_n rs_n, bias_n))   (bias_n = 0 without a bias).
// Per-tile row and column scales are staged in LDS during the prologue (RingScales).
template <int BM, int BN>
struct RingScales {
  // floats: rowA[BM] (alpha_m / 16), rowB[BM] (beta_m; 8-bit codes: beta_m + 128 alpha_m),
  // colS[BN] (s_n), colR[BN] (rs_n), colB[BN] (bias_n)
  static constexpr int COUNT = 2 * BM + 3 * BN;
  static constexpr int BYTES = COUNT * 4;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, static_cast<int>(bytes), 0x00020000);
}

// Scale value `idx` of a tile (RingScales layout), in two steps: fetch() reads every
// candidate source at a clamped index, unconditionally, and value() selects and converts.
// The caller issues the fetches before the tile's first copies and calls value() after the
// first stage has landed: the loads are then all in flight at once and off the copies'
// path (loads in branches made the compiler wait for each before the copies went out).
// Out-of-range rows/columns give 0.
struct ScaleFetch {
  float xa, xb, wa;
  int32_t rs;
  uint16_t bias;
};
template <int BM, int BN>
__device__ __forceinline__ ScaleFetch scale_fetch(const GemmArgs& g, int idx, int64_t m0, int64_t n0) {
  const int t = idx < 2 * BM ? 0 : idx - 2 * BM;
  const int64_t m = m0 + (idx % BM), n = n0 + (t % BN);
  const int64_t mc = m < g.M ? m : g.M - 1, nc = n < g.N ? n : g.N - 1;
  // without a bias the fetch reads (and discards) the first bytes of the scales
  const uint16_t* bp = g.bias ? g.bias : reinterpret_cast<const uint16_t*>(g.wa);
  return ScaleFetch{g.xa[mc], g.xb[mc], g.wa[nc], g.rs[nc], bp[nc]};
}
template <int BM, int BN>
__device__ __forceinline__ float scale_value(const GemmArgs& g, const ScaleFetch& f, int idx, int64_t m0, int64_t n0) {
  if (idx < 2 * BM) {
    if (m0 + (idx % BM) >= g.M) return 0.0f;
    if (idx < BM) return __fmul_rn(f.xa, 0.0625f);
    return g.a8 ? __fmaf_rn(128.0f, f.xa, f.xb) : f.xb;  // 8-bit codes enter as qa - 128
  }
  const int t = idx - 2 * BM;
  if (n0 + (t % BN) >= g.N) return 0.0f;
  if (t < BN) return f.wa;
  if (t < 2 * BN) return static_cast<float>(f.rs);
  return g.bias ? h2f(f.bias) : 0.0f;
}

// Fast path: the wave's columns lie inside N, rows past M are dropped by the buffer range,
// output rows are 8-byte aligned and the output fits a 31-bit byte range.
// Byte address in a staged output tile (rows of RB bytes, 16-byte chunks of row r XOR-ed
// with r % (RB / 16) so that the 32 rows one store instruction spans fall on different banks).
template <int RB>
__device__ __forceinline__ uint32_t stage_addr(int r, int b) {
  constexpr int CH = RB / 16;
  return static_cast<uint32_t>(r * RB + (((b >> 4) ^ (r & (CH - 1))) << 4) + (b & 15));
}

// Stores a staged BM x BNO fp16 output tile (rows m0.., columns n0o..) with whole-row 16-byte
// pieces: one store instruction covers 64 / (BNO / 8) full rows.  Rows past M are dropped by
// the buffer range.  Needs ldy % 8 == 0, a 16-byte aligned y and n0o % 8 == 0.
template <int BM, int BNO>
__device__ __forceinline__ void store_staged(const GemmArgs& g, const uint8_t* stg, int64_t m0, int64_t n0o, int wave,
                                             int waves, int lane) {
  constexpr int RB = BNO * 2, CH = RB / 16, RPI = 64 / CH;
  static_assert(CH <= 64 && 64 % CH == 0, "rows of at most 1 KB");
  const __amdgpu_buffer_rsrc_t ry = buf_rsrc(g.y, g.M * g.ldy * 2);
  const int k = lane % CH;
  for (int r0 = wave * RPI; r0 < BM; r0 += waves * RPI) {
    const int rr = r0 + lane / CH;
    const v4u v = *reinterpret_cast<const v4u*>(stg + stage_addr<RB>(rr, 16 * k));
    const int64_t m = m0 + rr;
    const uint32_t off = m < g.M ? static_cast<uint32_t>((m * g.ldy + n0o) * 2 + 16 * k) : 0x80000000u;
    __builtin_amdgcn_raw_buffer_store_b128(v, ry, static_cast<int>(off), 0, 0);
  }
}

template <int TM, int TN, int BM, int BN>
__device__ __forceinline__ void ring_epilogue_fast(const GemmArgs& g, const v16i (&acc)[TM][TN], int64_t mw, int64_t nw,
                                                   int tm, int tn, int lane, const float* __restrict__ sc) {
  const int c = lane & 31;
  const int h = lane >> 5;
  const float* rowA = sc;
  const float* rowB = sc + BM;
  const float* colS = sc + 2 * BM;
  const float* colR = colS + BN;
  const float* colB = colR + BN;
  const __amdgpu_buffer_rsrc_t ry = buf_rsrc(g.y, g.M * g.ldy * 2);
  float ra[TM], rb[TM];
  uint32_t yo[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = (tm + i) * 32 + c;
    ra[i] = rowA[r];
    rb[i] = rowB[r];
    const int64_t m = mw + i * 32 + c;
    yo[i] = m < g.M ? static_cast<uint32_t>((m * g.ldy + nw + 4 * h) * 2) : 0x80000000u;
  }
  // column scales of all TN blocks first, then the stores row block by row block, so that
  // the TN * 64 bytes a lane half writes per row go out in consecutive instructions (whole
  // 128-byte lines reach L2 together instead of halves written back separately)
  float s[TN][16], w[TN][16], bv[TN][16];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int cb = (tn + j) * 32 + 8 * q + 4 * h;
      const float4 sv = *reinterpret_cast<const float4*>(colS + cb);
      const float4 rv = *reinterpret_cast<const float4*>(colR + cb);
      const float4 bb = *reinterpret_cast<const float4*>(colB + cb);
      const float s4[4] = {sv.x, sv.y, sv.z, sv.w}, r4[4] = {rv.x, rv.y, rv.z, rv.w}, b4[4] = {bb.x, bb.y, bb.z, bb.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s[j][4 * q + e] = s4[e];
        w[j][4 * q + e] = __fmul_rn(s4[e], r4[e]);
        bv[j][4 * q + e] = b4[e];
      }
    }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        uint32_t pk[2];
#pragma unroll
        for (int e2 = 0; e2 < 2; ++e2) {
          float yv[2];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int r = 4 * q + 2 * e2 + u;
            const float t = __fmul_rn(s[j][r], static_cast<float>(acc[i][j][r]));
            yv[u] = fp32_result(__fmaf_rn(ra[i], t, __fmaf_rn(rb[i], w[j][r], bv[j][r])));  // bias 0 without one
          }
          pk[e2] = f2h2(yv[0], yv[1]);
        }
        __builtin_amdgcn_raw_buffer_store_b64(v2u{pk[0], pk[1]}, ry, static_cast<int>(yo[i] + (j * 32 + 8 * q) * 2), 0, 0);
      }
    }
  }
}

// Checked path: edge tiles, unaligned or large outputs, and the raw accumulator output.
template <int TM, int TN, int BM, int BN>
__device__ __forceinline__ void ring_epilogue_checked(const GemmArgs& g, const v16i (&acc)[TM][TN], int64_t mw,
                                                      int64_t nw, int tm, int tn, int lane, const float* __restrict__ sc) {
  const int c = lane & 31;
  const int h = lane >> 5;
  const float* rowA = sc;
  const float* rowB = sc + BM;
  const float* colS = sc + 2 * BM;
  const float* colR = colS + BN;
  const float* colB = colR + BN;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int64_t m = mw + i * 32 + c;
    if (m >= g.M) continue;
    const float ra = rowA[(tm + i) * 32 + c], rb = rowB[(tm + i) * 32 + c];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int cl = (tn + j) * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        const int64_t n = nw + j * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (n >= g.N) continue;
        const float s = colS[cl];
        const float t = __fmul_rn(s, static_cast<float>(acc[i][j][r]));
        const float yv = fp32_result(__fmaf_rn(ra, t, __fmaf_rn(rb, __fmul_rn(s, colR[cl]), colB[cl])));
        g.y[m * g.ldy + n] = f2h(yv);
        if (g.dbg_acc) g.dbg_acc[m * g.N + n] = (acc[i][j][r] >> 4) + (g.a8 ? 128 * g.rs[n] : 0);
      }
    }
  }
}

// SiLU(gate) * up of two dequantised fp32 outputs, as the fp16 input of down_proj:
// g u / (1 + e^-g), the quotient as a product with v_rcp_f32 (1 ulp; the result is rounded
// to fp16) instead of the IEEE division sequence, which took most of the gate/up epilogue's
// instructions; for g -> -inf the denominator is +inf, its reciprocal 0 and the product 0.
__device__ __forceinline__ float swiglu_value(float gv, float uv) {
  return __fmul_rn(__fmul_rn(gv, uv), __builtin_amdgcn_rcpf(__fadd_rn(1.0f, __expf(-gv))));
}

// Gate/up epilogues: wq interleaves gate and up rows in blocks of 32, so the wave's block
// pair (2p, 2p + 1) holds the gate and up outputs of the same 32 columns in the same lane
// and registers; output column = (interleaved column of the gate block) / 2 + offset.
template <int TM, int TN, int BM, int BN>
__device__ __forceinline__ void ring_epilogue_swiglu_fast(const GemmArgs& g, const v16i (&acc)[TM][TN], int64_t mw,
                                                          int64_t nw, int tm, int tn, int lane,
                                                          const float* __restrict__ sc) {
  static_assert(TN % 2 == 0, "gate/up block pairs");
  const int c = lane & 31;
  const int h = lane >> 5;
  const float* rowA = sc;
  const float* rowB = sc + BM;
  const float* colS = sc + 2 * BM;
  const float* colR = colS + BN;
  const float* colB = colR + BN;
  const __amdgpu_buffer_rsrc_t ry = buf_rsrc(g.y, g.M * g.ldy * 2);
  float ra[TM], rb[TM];
  uint32_t yo[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = (tm + i) * 32 + c;
    ra[i] = rowA[r];
    rb[i] = rowB[r];
    const int64_t m = mw + i * 32 + c;
    yo[i] = m < g.M ? static_cast<uint32_t>((m * g.ldy + nw / 2 + 4 * h) * 2) : 0x80000000u;
  }
  float s[TN][16], w[TN][16], bv[TN][16];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int cb = (tn + j) * 32 + 8 * q + 4 * h;
      const float4 sv = *reinterpret_cast<const float4*>(colS + cb);
      const float4 rv = *reinterpret_cast<const float4*>(colR + cb);
      const float4 bb = *reinterpret_cast<const float4*>(colB + cb);
      const float s4[4] = {sv.x, sv.y, sv.z, sv.w}, r4[4] = {rv.x, rv.y, rv.z, rv.w}, b4[4] = {bb.x, bb.y, bb.z, bb.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s[j][4 * q + e] = s4[e];
        w[j][4 * q + e] = __fmul_rn(s4[e], r4[e]);
        bv[j][4 * q + e] = b4[e];
      }
    }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
#pragma unroll
      for (int p = 0; p < TN / 2; ++p) {
        uint32_t pk[2];
#pragma unroll
        for (int e2 = 0; e2 < 2; ++e2) {
          float hv[2];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int r = 4 * q + 2 * e2 + u;
            const int jg = 2 * p, ju = 2 * p + 1;
            const float tg = __fmul_rn(s[jg][r], static_cast<float>(acc[i][jg][r]));
            const float tu = __fmul_rn(s[ju][r], static_cast<float>(acc[i][ju][r]));
            const float gv = fp32_result(__fmaf_rn(ra[i], tg, __fmaf_rn(rb[i], w[jg][r], bv[jg][r])));
            const float uv = fp32_result(__fmaf_rn(ra[i], tu, __fmaf_rn(rb[i], w[ju][r], bv[ju][r])));
            hv[u] = fp32_result(swiglu_value(gv, uv));
          }
          pk[e2] = f2h2(hv[0], hv[1]);
        }
        __builtin_amdgcn_raw_buffer_store_b64(v2u{pk[0], pk[1]}, ry, static_cast<int>(yo[i] + (p * 32 + 8 * q) * 2), 0, 0);
      }
    }
  }
}

template <int TM, int TN, int BM, int BN>
__device__ __forceinline__ void ring_epilogue_swiglu_checked(const GemmArgs& g, const v16i (&acc)[TM][TN],
                                                             int64_t mw, int64_t nw, int tm, int tn, int lane,
                                                             const float* __restrict__ sc) {
  static_assert(TN % 2 == 0, "gate/up block pairs");
  const int c = lane & 31;
  const int h = lane >> 5;
  const float* rowA = sc;
  const float* rowB = sc + BM;
  const float* colS = sc + 2 * BM;
  const float* colR = colS + BN;
  const float* colB = colR + BN;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int64_t m = mw + i * 32 + c;
    if (m >= g.M) continue;
    const float ra = rowA[(tm + i) * 32 + c], rb = rowB[(tm + i) * 32 + c];
#pragma unroll
    for (int p = 0; p < TN / 2; ++p) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int off = 8 * (r >> 2) + 4 * h + (r & 3);
        const int cg = (tn + 2 * p) * 32 + off, cu = cg + 32;
        const int64_t ng = nw + 64 * p + off;  // gate column; its up column ng + 32 < N (N % 64 == 0)
        if (ng >= g.N) continue;
        const float gv = fp32_result(__fmaf_rn(ra, __fmul_rn(colS[cg], static_cast<float>(acc[i][2 * p][r])),
                                               __fmaf_rn(rb, __fmul_rn(colS[cg], colR[cg]), colB[cg])));
        const float uv = fp32_result(__fmaf_rn(ra, __fmul_rn(colS[cu], static_cast<float>(acc[i][2 * p + 1][r])),
                                               __fmaf_rn(rb, __fmul_rn(colS[cu], colR[cu]), colB[cu])));
        g.y[m * g.ldy + (nw + 64 * p) / 2 + off] = f2h(fp32_result(swiglu_value(gv, uv)));
      }
    }
  }
}

// Epilogue of a ring-kernel block: plain or gate/up, vector (fast) or element-wise stores.
// The fast epilogue through a staged tile in LDS (stg: BM x BN fp16, or BM x BN/2 for
// gate/up, in the ring's bytes, which the caller has drained): every wave writes its block
// (same arithmetic as the other epilogues), a workgroup barrier, then the whole tile goes
// out in whole-row pieces.  Column groups q run outermost so that only one group's column
// scales are live.  Needs what store_staged needs.
template <int TM, int TN, int BM, int BN>
__device__ __forceinline__ void ring_epilogue_staged(const GemmArgs& g, const v16i (&acc)[TM][TN], int64_t m0,
                                                     int64_t n0, int tm, int tn, int lane, const float* __restrict__ sc,
                                                     uint8_t* stg, int wave, int waves) {
  const int c = lane & 31;
  const int h = lane >> 5;
  const float* rowA = sc;
  const float* rowB = sc + BM;
  const float* colS = sc + 2 * BM;
  const float* colR = colS + BN;
  const float* colB = colR + BN;
  float ra[TM], rb[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    ra[i] = rowA[(tm + i) * 32 + c];
    rb[i] = rowB[(tm + i) * 32 + c];
  }
  const bool sw = g.swiglu;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float s[TN][4], w[TN][4], bv[TN][4];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int cb = (tn + j) * 32 + 8 * q + 4 * h;
      const float4 sv = *reinterpret_cast<const float4*>(colS + cb);
      const float4 rv = *reinterpret_cast<const float4*>(colR + cb);
      const float4 bb = *reinterpret_cast<const float4*>(colB + cb);
      const float s4[4] = {sv.x, sv.y, sv.z, sv.w}, r4[4] = {rv.x, rv.y, rv.z, rv.w}, b4[4] = {bb.x, bb.y, bb.z, bb.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s[j][e] = s4[e];
        w[j][e] = __fmul_rn(s4[e], r4[e]);
        bv[j][e] = b4[e];
      }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r0 = 4 * q;
      const int row = (tm + i) * 32 + c;
      if (sw) {
        if constexpr (TN % 2 == 0) {
#pragma unroll
          for (int p = 0; p < TN / 2; ++p) {
            uint32_t pk[2];
#pragma unroll
            for (int e2 = 0; e2 < 2; ++e2) {
              float hv[2];
#pragma unroll
              for (int u = 0; u < 2; ++u) {
                const int e = 2 * e2 + u;
                const int jg = 2 * p, ju = 2 * p + 1;
                const float tg = __fmul_rn(s[jg][e], static_cast<float>(acc[i][jg][r0 + e]));
                const float tu = __fmul_rn(s[ju][e], static_cast<float>(acc[i][ju][r0 + e]));
                const float gv = fp32_result(__fmaf_rn(ra[i], tg, __fmaf_rn(rb[i], w[jg][e], bv[jg][e])));
                const float uv = fp32_result(__fmaf_rn(ra[i], tu, __fmaf_rn(rb[i], w[ju][e], bv[ju][e])));
                hv[u] = fp32_result(swiglu_value(gv, uv));
              }
              pk[e2] = f2h2(hv[0], hv[1]);
            }
            *reinterpret_cast<v2u*>(stg + stage_addr<BN>(row, ((tn / 2 + p) * 32 + 8 * q + 4 * h) * 2)) =
                v2u{pk[0], pk[1]};
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          uint32_t pk[2];
#pragma unroll
          for (int e2 = 0; e2 < 2; ++e2) {
            float yv[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              const int e = 2 * e2 + u;
              const float t = __fmul_rn(s[j][e], static_cast<float>(acc[i][j][r0 + e]));
              yv[u] = fp32_result(__fmaf_rn(ra[i], t, __fmaf_rn(rb[i], w[j][e], bv[j][e])));
            }
            pk[e2] = f2h2(yv[0], yv[1]);
          }
          *reinterpret_cast<v2u*>(stg + stage_addr<BN * 2>(row, ((tn + j) * 32 + 8 * q + 4 * h) * 2)) =
              v2u{pk[0], pk[1]};
        }
      }
    }
  }
  __syncthreads();
  if (sw)
    store_staged<BM, BN / 2>(g, stg, m0, n0 / 2, wave, waves, lane);
  else
    store_staged<BM, BN>(g, stg, m0, n0, wave, waves, lane);
}

template <int TM, int TN, int BM, int BN>
__device__ __forceinline__ void ring_epilogue(const GemmArgs& g, const v16i (&acc)[TM][TN], int64_t mw, int64_t nw,
                                              int tm, int tn, int lane, const float* __restrict__ sc, bool fast) {
  if (g.swiglu) {
    if constexpr (TN % 2 == 0) {
      if (fast)
        ring_epilogue_swiglu_fast<TM, TN, BM, BN>(g, acc, mw, nw, tm, tn, lane, sc);
      else
        ring_epilogue_swiglu_checked<TM, TN, BM, BN>(g, acc, mw, nw, tm, tn, lane, sc);
    }
    return;
  }
  if (fast)
    ring_epilogue_fast<TM, TN, BM, BN>(g, acc, mw, nw, tm, tn, lane, sc);
  else
    ring_epilogue_checked<TM, TN, BM, BN>(g, acc, mw, nw, tm, tn, lane, sc);
}

// ------------------------------------------------------------------ prefill tile kernel
constexpr int kBKB = 64;               // packed bytes per row per stage (128 k)
constexpr int kPitch = 72;             // LDS row pitch (bytes)

template <int TM, int TN>
struct Frags {
  uint2 a[TM];
  uint2 b[TN];
};

template <int TM, int TN>
__device__ __forceinline__ void read_frags(Frags<TM, TN>& f, const uint8_t* As, const uint8_t* Bs, int wm, int wn,
                                           int frow, int off) {
#pragma unroll
  for (int i = 0; i < TM; ++i) f.a[i] = *reinterpret_cast<const uint2*>(As + (wm + i * 32 + frow) * kPitch + off);
#pragma unroll
  for (int j = 0; j < TN; ++j) f.b[j] = *reinterpret_cast<const uint2*>(Bs + (wn + j * 32 + frow) * kPitch + off);
}

// TM x TN MFMAs of one 32-k step; the expansion of the next step's fragments (read from
// LDS before these MFMAs) is interleaved with them.
template <int TM, int TN>
__device__ __forceinline__ void mma_step(v16i (&acc)[TM][TN], const v4i (&af)[TM], const v4i (&bf)[TN],
                                         v4i (&naf)[TM], v4i (&nbf)[TN], const Frags<TM, TN>& nf, bool expand_next) {
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
  if (expand_next) {
#pragma unroll
    for (int i = 0; i < TM; ++i) naf[i] = expand_act(nf.a[i]);
#pragma unroll
    for (int j = 0; j < TN; ++j) nbf[j] = expand_wgt(nf.b[j]);
  }
  constexpr int NM = TM * TN;
  constexpr int NV = 6 * (TM + TN);
  constexpr int PER = (NV + NM - 3) / (NM - 2);
  __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
#pragma unroll
  for (int k = 0; k < NM - 2; ++k) {
    __builtin_amdgcn_sched_group_barrier(0x002, PER, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  }
}

// WAVES_M x WAVES_N waves per workgroup, each owning TM x TN MFMA blocks of 32 x 32.
template <int WAVES_M, int WAVES_N, int TM, int TN>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N)
w4a4_gemm_tile(GemmArgs g) {
  constexpr int THREADS = 64 * WAVES_M * WAVES_N;
  constexpr int BM = WAVES_M * TM * 32;
  constexpr int BN = WAVES_N * TN * 32;
  constexpr int kStage = (BM + BN) * kPitch;
  constexpr int kAChunks = BM * 4 / THREADS;  // 16-byte chunks per thread per stage
  constexpr int kBChunks = BN * 4 / THREADS;
  static_assert(kAChunks * THREADS == BM * 4 && kBChunks * THREADS == BN * 4, "staging split");
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * kStage];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  int64_t m0, n0;
  tile_origin(BM, BN, m0, n0);
  const int wm = (wave / WAVES_N) * (TM * 32);
  const int wn = (wave % WAVES_N) * (TN * 32);
  const int64_t KB = g.K / 2;
  const int nstage = static_cast<int>((KB + kBKB - 1) / kBKB);

  // Staging: chunk index c = tid + q*THREADS covers tile row (c % 16) + 16 (c / 64) and
  // 16-byte column (c / 16) % 4, so 16 consecutive lanes write 16 rows of one column (at
  // the 72-byte pitch those hit distinct bank pairs).  Rows past M or N are clamped to the
  // last valid row: they only feed outputs that are never stored.  Columns past K (a half
  // stage when K % 128 == 64) are zeroed on the A side, so they contribute nothing.
  const int64_t ma = g.M - 1, nb = g.N - 1;
  const int srow = (tid & 15) + 16 * (tid >> 6);  // tile row of chunk q = 0; chunk q adds q * THREADS / 4
  const int scol = ((tid >> 4) & 3) * 16;
  uint4 ra[kAChunks], rb[kBChunks];
  auto gload = [&](int st) {
    const int64_t kb = static_cast<int64_t>(st) * kBKB;
    const bool kok = kb + scol < KB;
    // a chunk past K (the second half of the last stage when K % 128 == 64) reads column
    // scol of stage 0 instead, for both operands, so every load stays inside its row; the
    // A chunk is then zeroed and the product adds nothing
    const int64_t ka = (kok ? kb : 0) + scol;
#pragma unroll
    for (int q = 0; q < kAChunks; ++q) {
      const int64_t r = m0 + srow + q * (THREADS / 4);
      const uint4 v = *reinterpret_cast<const uint4*>(g.xq + (r < ma ? r : ma) * KB + ka);
      ra[q] = kok ? v : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < kBChunks; ++q) {
      const int64_t r = n0 + srow + q * (THREADS / 4);
      rb[q] = *reinterpret_cast<const uint4*>(g.wq + (r < nb ? r : nb) * KB + ka);
    }
  };
  auto lstore = [&](int buf) {
    uint8_t* base = lds + buf * kStage + srow * kPitch + scol;
#pragma unroll
    for (int q = 0; q < kAChunks; ++q) {
      uint8_t* p = base + q * (THREADS / 4) * kPitch;
      *reinterpret_cast<uint2*>(p) = make_uint2(ra[q].x, ra[q].y);
      *reinterpret_cast<uint2*>(p + 8) = make_uint2(ra[q].z, ra[q].w);
    }
#pragma unroll
    for (int q = 0; q < kBChunks; ++q) {
      uint8_t* p = base + (BM + q * (THREADS / 4)) * kPitch;
      *reinterpret_cast<uint2*>(p) = make_uint2(rb[q].x, rb[q].y);
      *reinterpret_cast<uint2*>(p + 8) = make_uint2(rb[q].z, rb[q].w);
    }
  };

  v16i acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0;

  const int frow = lane & 31;
  const int fofs = (lane >> 5) * 8;
  gload(0);
  lstore(0);
  __syncthreads();
  v4i af0[TM], bf0[TN], af1[TM], bf1[TN];
  Frags<TM, TN> f;
  read_frags(f, lds, lds + BM * kPitch, wm, wn, frow, fofs);
#pragma unroll
  for (int i = 0; i < TM; ++i) af0[i] = expand_act(f.a[i]);
#pragma unroll
  for (int j = 0; j < TN; ++j) bf0[j] = expand_wgt(f.b[j]);

  for (int st = 0; st < nstage; ++st) {
    const int buf = st & 1;
    const bool more = st + 1 < nstage;
    if (more) gload(st + 1);
    const uint8_t* As = lds + buf * kStage;
    const uint8_t* Bs = As + BM * kPitch;
    // k-steps 0..3 of this stage, ping-ponging the expanded fragments
    read_frags(f, As, Bs, wm, wn, frow, 16 + fofs);
    mma_step(acc, af0, bf0, af1, bf1, f, true);
    read_frags(f, As, Bs, wm, wn, frow, 32 + fofs);
    mma_step(acc, af1, bf1, af0, bf0, f, true);
    read_frags(f, As, Bs, wm, wn, frow, 48 + fofs);
    mma_step(acc, af0, bf0, af1, bf1, f, true);
    if (more) lstore(buf ^ 1);
    __syncthreads();
    if (more) read_frags(f, lds + (buf ^ 1) * kStage, lds + (buf ^ 1) * kStage + BM * kPitch, wm, wn, frow, fofs);
    mma_step(acc, af1, bf1, af0, bf0, f, more);
  }

  tile_epilogue(g, acc, m0 + wm, n0 + wn, lane);
}

// ------------------------------------------------------------------ LDS-ring tile kernel
// Packed operand tiles go from global memory straight into LDS (buffer_load_dwordx4 ... lds:
// no registers, no VALU), NS stages deep, so a stage's loads are in flight for NS - 1 stages
// of MFMA work.  A stage covers 128 k (64 packed bytes per row) and is laid out as 1 KB
// blocks, one per 32 rows and pair of 16-byte chunks: lane l of the copying wave brings row
// l % 32, chunk 2p + l / 32 to byte 16 l of the block.  A wave reads a block back with one
// contiguous ds_read_b128 (no bank conflicts); each lane then holds 32 codes of one row,
// which expand into the operands of two MFMA k-steps.  Both operands use the same k-slot
// order, so the dot product is unchanged.  Rows past M or N and chunks past K are out of the
// buffer range and land as zeros.
// 8-bit activations (A8, the W4A8 setting): a stage row is 128 code bytes, 8 chunks, and the
// A blocks are one per 32 rows and (chunk pair p, half H): lane l of the copying wave brings
// row l % 32, chunk 4p + 2(l / 32) + H, so the lane (c, h) that reads it back holds exactly
// the 16 codes of k-step (p, H) that the 4-bit expansion gives it (k = 64p + 32h + 16H + e);
// v_perm_b32 puts them in the same slot order and an xor with 0x80 makes them signed.
template <int WAVES_M, int WAVES_N, int TM, int TN, int NS, bool A8 = false>
struct Ring {
  static constexpr int WAVES = WAVES_M * WAVES_N;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int BM = WAVES_M * TM * 32;
  static constexpr int BN = WAVES_N * TN * 32;
  static constexpr int ABLK = BM / (A8 ? 8 : 16);  // 1 KB blocks per stage: 32 rows x 2 (A8: 4) chunk pairs
  static constexpr int BBLK = BN / 16;
  static constexpr int ADPW = ABLK / WAVES;  // block copies per wave per stage
  static constexpr int DPW = (ABLK + BBLK) / WAVES;
  static constexpr int STAGE = (ABLK + BBLK) * 1024;
  static_assert(ADPW * WAVES == ABLK && DPW * WAVES == ABLK + BBLK, "blocks split evenly over waves");
  static_assert(NS >= 2 && (NS - 1) * DPW <= 63, "outstanding copies fit the vmcnt counter");
};

template <int TM, int TN, bool A8 = false>
struct RingPacked {  // one chunk pair (two k-steps) of the wave's A and B blocks
  v4u a[TM][A8 ? 2 : 1];
  v4u b[TN];
};

// 16 8-bit activation codes k0..k15 (natural order) -> signed operand in the slot order of
// the nibble expansion (k0 k2 k4 k6 | k1 k3 k5 k7 | k8 ...)
__device__ __forceinline__ v4i act8_operand(const v4u d) {
  const uint32_t f = 0x80808080u;
  return v4i{static_cast<int>(__builtin_amdgcn_perm(d[1], d[0], 0x06040200u) ^ f),
             static_cast<int>(__builtin_amdgcn_perm(d[1], d[0], 0x07050301u) ^ f),
             static_cast<int>(__builtin_amdgcn_perm(d[3], d[2], 0x06040200u) ^ f),
             static_cast<int>(__builtin_amdgcn_perm(d[3], d[2], 0x07050301u) ^ f)};
}
template <int TM, int TN>
struct RingOps {  // MFMA operands of one k-step
  v4i a[TM];
  v4i b[TN];
};

// Operands of k-step H (0: dwords 0-1, 1: dwords 2-3) of a packed chunk pair.
template <int H, int TM, int TN, bool A8>
__device__ __forceinline__ void expand_half(const RingPacked<TM, TN, A8>& P, RingOps<TM, TN>& E) {
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    if constexpr (A8) {
      E.a[i] = act8_operand(P.a[i][H]);
    } else {
      const uint32_t d0 = P.a[i][0][2 * H], d1 = P.a[i][0][2 * H + 1];
      E.a[i] = v4i{static_cast<int>(d0 & 0x0F0F0F0Fu), static_cast<int>((d0 >> 4) & 0x0F0F0F0Fu),
                   static_cast<int>(d1 & 0x0F0F0F0Fu), static_cast<int>((d1 >> 4) & 0x0F0F0F0Fu)};
    }
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const uint32_t d0 = P.b[j][2 * H], d1 = P.b[j][2 * H + 1];
    E.b[j] = v4i{static_cast<int>((d0 << 4) & 0xF0F0F0F0u), static_cast<int>(d0 & 0xF0F0F0F0u),
                 static_cast<int>((d1 << 4) & 0xF0F0F0F0u), static_cast<int>(d1 & 0xF0F0F0F0u)};
  }
}

// s_waitcnt with vmcnt = VM (0..63: bits 3:0 and 15:14) and lgkmcnt = 0 (expcnt not waited on)
template <int VM>
__device__ __forceinline__ void wait_vm_lgkm0() {
  static_assert(VM >= 0 && VM <= 63, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt((VM & 0xF) | ((VM >> 4) << 14) | (0x7 << 4));
}

// LDS of a ring kernel with KS groups of waves splitting K: one ring per group (reused at
// the end for the groups' exchange of partial sums), then the tile's epilogue scales.
template <int WAVES_M, int WAVES_N, int TM, int TN, int NS, int KS, bool A8 = false>
struct RingLds {
  using R = Ring<WAVES_M, WAVES_N, TM, TN, NS, A8>;
  static constexpr int RINGS = KS * NS * R::STAGE;
  static constexpr int XCH = KS == 1 ? 0 : KS * R::WAVES * (TM / 2) * TN * 16 * 64 * 4;
  static constexpr int SCALES = RINGS > XCH ? RINGS : XCH;  // byte offset of the scales
  static constexpr int BYTES = SCALES + RingScales<R::BM, R::BN>::BYTES;
};

// KS = 2: two groups of WAVES_M x WAVES_N waves share the tile and split its k-stages in
// two halves, each group with its own ring (twice the waves per SIMD when the tile count
// leaves the CUs one workgroup each).  At the end each group hands the other the int32
// partial sums of the half of its block that the other finishes (through LDS; integer
// sums, so the result is bit-identical to KS = 1), and each finishes half of the rows.
template <int WAVES_M, int WAVES_N, int TM, int TN, int NS, int WPE, int KS, bool A8 = false>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N * KS, WPE)
w4a4_gemm_ring(GemmArgs g) {
  using R = Ring<WAVES_M, WAVES_N, TM, TN, NS, A8>;
  using L = RingLds<WAVES_M, WAVES_N, TM, TN, NS, KS, A8>;
  using SC = RingScales<R::BM, R::BN>;
  static_assert(KS == 1 || (KS == 2 && TM % 2 == 0), "K split of two needs an even TM");
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  float* const scales = reinterpret_cast<float*>(lds + L::SCALES);
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = wid / R::WAVES;   // K slice of this wave's group
  const int wave = wid % R::WAVES;  // wave within the group
  uint8_t* const ring = lds + grp * NS * R::STAGE;
  int64_t m0, n0;
  tile_origin(R::BM, R::BN, m0, n0);
  const int wm = (wave / WAVES_N) * TM;  // first 32-row group of this wave in the tile
  const int wn = (wave % WAVES_N) * TN;
  const uint32_t KB = static_cast<uint32_t>(g.K / 2);
  const uint32_t KA = A8 ? 2 * KB : KB;  // activation bytes per row
  // stages per group; the group's stage st is stage st0 + st of the whole K (past K: zeros)
  const int nstage = static_cast<int>(((KB + 63) / 64 + KS - 1) / KS);
  const uint32_t st0 = static_cast<uint32_t>(grp * nstage);

  // Buffer ranges: offsets are 32-bit and (M + BM) * KA < 2^31 is checked on the host.
  const __amdgpu_buffer_rsrc_t rsa =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(g.xq), 0, static_cast<int>(g.M * KA), 0x00020000);
  const __amdgpu_buffer_rsrc_t rsb =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(g.wq), 0, static_cast<int>(g.N * KB), 0x00020000);
  // Copy d of this wave is block b = wave + WAVES d of a stage: A blocks first, then B.
  uint32_t rowoff[R::DPW], colofs[R::DPW];
  static_for<R::DPW>([&](auto dc) {
    constexpr int d = decltype(dc)::value;
    const int b = wave + R::WAVES * d;
    const int bl = d < R::ADPW ? b : b - R::ABLK;
    if (A8 && d < R::ADPW) {  // block (row group, p, H): chunk 4p + 2h + H of the 128-byte row
      const int64_t row = m0 + (bl >> 2) * 32 + (lane & 31);
      rowoff[d] = static_cast<uint32_t>(row) * KA;
      colofs[d] = ((bl >> 1) & 1) * 64 + (lane >> 5) * 32 + (bl & 1) * 16;
    } else {
      const int64_t row = (d < R::ADPW ? m0 : n0) + (bl >> 1) * 32 + (lane & 31);
      rowoff[d] = static_cast<uint32_t>(row) * KB;
      colofs[d] = (bl & 1) * 32 + (lane >> 5) * 16;
    }
  });
  auto issue = [&](int st) {
    uint8_t* sb = ring + (st % NS) * R::STAGE;
    const uint32_t k0 = (st0 + static_cast<uint32_t>(st)) * 64;
    const bool live = st < nstage;
    static_for<R::DPW>([&](auto dc) {
      constexpr int d = decltype(dc)::value;
      constexpr bool a8blk = A8 && d < R::ADPW;
      const uint32_t col = (a8blk ? 2 * k0 : k0) + colofs[d];
      // past K, or a stage past the group's end (issued only to keep the copy count
      // uniform; it may lie in the next group's slice): out of range, lands as zeros
      const uint32_t off = (live && col < (a8blk ? KA : KB)) ? rowoff[d] + col : 0x80000000u;
      auto* dst = reinterpret_cast<__attribute__((address_space(3))) void*>(
          reinterpret_cast<uintptr_t>(sb + (wave + R::WAVES * d) * 1024));
      if constexpr (d < R::ADPW)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, dst, 16, static_cast<int>(off), 0, 0, 0);
      else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, dst, 16, static_cast<int>(off), 0, 0, 0);
    });
  };
  auto read = [&](RingPacked<TM, TN, A8>& P, int st, int p) {
    const uint8_t* sb = ring + (st % NS) * R::STAGE + lane * 16;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      if constexpr (A8) {
        P.a[i][0] = *reinterpret_cast<const v4u*>(sb + (wm + i) * 4096 + (2 * p) * 1024);
        P.a[i][1] = *reinterpret_cast<const v4u*>(sb + (wm + i) * 4096 + (2 * p + 1) * 1024);
      } else {
        P.a[i][0] = *reinterpret_cast<const v4u*>(sb + (wm + i) * 2048 + p * 1024);
      }
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) P.b[j] = *reinterpret_cast<const v4u*>(sb + (R::ABLK + 2 * (wn + j) + p) * 1024);
  };
  // MFMAs of one k-step from E, with the next k-step's operands expanded into F in between
  constexpr int NM = TM * TN;
  constexpr int NV = (A8 ? 8 : 6) * TM + 6 * TN;
  constexpr int PER = (NV + NM - 2) / (NM - 1);
  auto mma = [&](v16i (&acc)[TM][TN], const RingOps<TM, TN>& E) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(E.b[j], E.a[i], acc[i][j], 0, 0, 0);
  };
  // ds_reads (NR of them) first, then one MFMA per PER expansion ops
  auto interleave = [&](auto nr) {
    constexpr int NR = decltype(nr)::value;
    if constexpr (NR > 0) __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
#pragma unroll
    for (int k = 0; k < NM - 1; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x002, PER, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
  };
  auto sync = [&]() {
    wait_vm_lgkm0<(NS - 2) * R::DPW>();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  v16i acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0;

  // Pipeline over k-steps (four per stage).  Packed chunk pairs are read from LDS two
  // k-steps before their first expansion, operands are expanded one k-step ahead of their
  // MFMAs, and the stage sync sits in the second k-step, after the last read of the
  // current stage's slot (which the copy issued right after it refills).
  // epilogue scales of the tile: loaded now, written to LDS after the first copies have
  // landed (the main loop's barriers publish them)
  constexpr int TT = R::THREADS * KS;
  constexpr int SPT = (SC::COUNT + TT - 1) / TT;
  ScaleFetch sf[SPT];
#pragma unroll
  for (int u = 0; u < SPT; ++u) {
    const int idx = static_cast<int>(threadIdx.x) + u * TT;
    sf[u] = scale_fetch<R::BM, R::BN>(g, idx < SC::COUNT ? idx : 0, m0, n0);
  }
  for (int s = 0; s < NS - 1; ++s) issue(s);
  sync();
#pragma unroll
  for (int u = 0; u < SPT; ++u) {
    const int idx = static_cast<int>(threadIdx.x) + u * TT;
    if (idx < SC::COUNT) scales[idx] = scale_value<R::BM, R::BN>(g, sf[u], idx, m0, n0);
  }
  issue(NS - 1);
  RingPacked<TM, TN, A8> P0, P1;
  RingOps<TM, TN> E0, E1;
  read(P0, 0, 0);
  read(P1, 0, 1);
  expand_half<0>(P0, E0);

  // Branch-free steady state: the last iteration also syncs, copies (out of range) and
  // expands the stage after the end; those operands are never used.
  for (int st = 0; st < nstage; ++st) {
    constexpr std::integral_constant<int, 0> none{};
    constexpr std::integral_constant<int, (A8 ? 2 : 1) * TM + TN> all{};  // ds_reads of one read()
    mma(acc, E0);                 // k-step 4 st
    expand_half<1>(P0, E1);
    interleave(none);
    sync();                       // stage st + 1 has landed; slot st is free
    issue(st + NS);
    read(P0, st + 1, 0);
    mma(acc, E1);                 // k-step 4 st + 1
    expand_half<0>(P1, E0);
    interleave(all);
    mma(acc, E0);                 // k-step 4 st + 2
    expand_half<1>(P1, E1);
    interleave(none);
    read(P1, st + 1, 1);
    mma(acc, E1);                 // k-step 4 st + 3
    expand_half<0>(P0, E0);
    interleave(all);
  }
  // copies of stages past the end may still be landing in LDS
  wait_vm_lgkm0<0>();
  asm volatile("" ::: "memory");

  // fast epilogue: the tile's columns inside N, 8-byte aligned output rows, 31-bit output range
  const bool fast = g.dbg_acc == nullptr && (g.ldy & 3) == 0 && (reinterpret_cast<uintptr_t>(g.y) & 7) == 0 &&
                    g.M * g.ldy * 2 < (int64_t{1} << 31) && n0 + R::BN <= g.N;
  if constexpr (KS == 1) {
    // whole-row stores through the drained ring when rows are 16-byte aligned (uniform over
    // the workgroup, as is the barrier inside)
    static_assert(R::BM * R::BN * 2 <= L::RINGS, "the output tile fits the ring");
    if (fast && (g.ldy & 7) == 0 && (reinterpret_cast<uintptr_t>(g.y) & 15) == 0) {
      __syncthreads();  // every wave's copies have landed and its last fragments are read
      ring_epilogue_staged<TM, TN, R::BM, R::BN>(g, acc, m0, n0, wm, wn, lane, scales, lds, wave, R::WAVES);
    } else {  // element-wise stores (a third, direct-store path would cost the kernel spills)
      ring_epilogue<TM, TN, R::BM, R::BN>(g, acc, m0 + wm * 32, n0 + wn * 32, wm, wn, lane, scales, false);
    }
  } else {
    // group h finishes row blocks [h*HT, h*HT + HT) of the wave's block
    constexpr int HT = TM / 2;
    constexpr int XW = HT * TN * 16;  // ints per lane handed over
    int* const xch = reinterpret_cast<int*>(lds);
    __builtin_amdgcn_s_barrier();  // both rings are drained and read for the last time
    asm volatile("" ::: "memory");
    auto put = [&](auto hc) {  // hand over half hc to the other group
      constexpr int h = decltype(hc)::value;
      int* dst = xch + (grp * R::WAVES + wave) * XW * 64 + lane;
#pragma unroll
      for (int i = 0; i < HT; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) dst[((i * TN + j) * 16 + r) * 64] = acc[h * HT + i][j][r];
    };
    auto take = [&](auto hc) {  // add the other group's partial sums of half hc
      constexpr int h = decltype(hc)::value;
      const int* src = xch + ((1 - grp) * R::WAVES + wave) * XW * 64 + lane;
#pragma unroll
      for (int i = 0; i < HT; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[h * HT + i][j][r] += src[((i * TN + j) * 16 + r) * 64];
    };
    auto finish = [&](auto hc) {
      constexpr int h = decltype(hc)::value;
      v16i part[HT][TN];
#pragma unroll
      for (int i = 0; i < HT; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) part[i][j] = acc[h * HT + i][j];
      const int64_t mw = m0 + (wm + h * HT) * 32, nw = n0 + wn * 32;
      ring_epilogue<HT, TN, R::BM, R::BN>(g, part, mw, nw, wm + h * HT, wn, lane, scales, fast);
    };
    constexpr std::integral_constant<int, 0> lo{};
    constexpr std::integral_constant<int, 1> hi{};
    if (grp == 0) put(hi); else put(lo);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (grp == 0) take(lo); else take(hi);
    if (grp == 0) finish(lo); else finish(hi);
  }
}

template <int WM, int WN, int TM, int TN, int NS, bool A8 = false>
bool fits_ring(const GemmArgs& g) {
  using R = Ring<WM, WN, TM, TN, NS, A8>;
  const int64_t kb = g.K / 2, ka = A8 ? g.K : kb;
  return (g.M + R::BM) * ka + 128 < (int64_t{1} << 31) && (g.N + R::BN) * kb + 64 < (int64_t{1} << 31);
}

// WPE: waves per SIMD the registers must allow (2 for two 4-wave workgroups per CU, or one
// workgroup of two K groups); KS: groups of waves splitting K.
template <int WM, int WN, int TM, int TN, int NS, int WPE = 1, int KS = 1, bool A8 = false>
hipError_t launch_ring(const GemmArgs& g, hipStream_t stream) {
  using R = Ring<WM, WN, TM, TN, NS, A8>;
  constexpr int LDS = RingLds<WM, WN, TM, TN, NS, KS, A8>::BYTES;
  static_assert(LDS <= 160 * 1024, "LDS of one CU");
  constexpr auto kern = w4a4_gemm_ring<WM, WN, TM, TN, NS, WPE, KS, A8>;
  const hipError_t init = set_max_lds<kern>(LDS);
  if (init != hipSuccess) return init;
  const dim3 grid(static_cast<unsigned>((g.N + R::BN - 1) / R::BN), static_cast<unsigned>((g.M + R::BM - 1) / R::BM));
  return launch(kern, grid, dim3(R::THREADS * KS), LDS, stream, g);
}

// Epilogue of one 16 x 16 block of a decode product (v_mfma_i32_16x16x64_i8 layout: lane
// r + 16 sg, register i holds D[4 sg + i][r]) for weight row n: the ring kernel's arithmetic
// (acc holds 16 x the sum; A8: of qa - 128, whose shift the zero-point term takes back).
template <bool A8>
__device__ __forceinline__ void decode_store(const GemmArgs& g, const v4i& acc, int64_t n, int sg) {
  if (n >= g.N) return;
  const float sn = g.wa[n];
  const float wn = __fmul_rn(sn, static_cast<float>(g.rs[n]));
  const float bn = g.bias ? h2f(g.bias[n]) : 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = 4 * sg + i;
    if (m >= g.M) continue;
    const float t = __fmul_rn(sn, static_cast<float>(acc[i]));
    const float xb = A8 ? __fmaf_rn(128.0f, g.xa[m], g.xb[m]) : g.xb[m];
    const float yv = fp32_result(__fmaf_rn(__fmul_rn(g.xa[m], 0.0625f), t, __fmaf_rn(xb, wn, bn)));
    g.y[m * g.ldy + n] = f2h(yv);
    if (g.dbg_acc) g.dbg_acc[m * g.N + n] = (acc[i] >> 4) + (A8 ? 128 * g.rs[n] : 0);
  }
}

// The same for a gate block (rows ng) and its up block (rows ng + 32): SiLU(g) u to output
// column col.
__device__ __forceinline__ void decode_store_swiglu(const GemmArgs& g, const v4i& accg, const v4i& accu, int64_t ng,
                                                    int64_t col, int sg) {
  if (ng >= g.N) return;
  const int64_t nu = ng + 32;
  const float scg = g.wa[ng], scu = g.wa[nu];
  const float wg = __fmul_rn(scg, static_cast<float>(g.rs[ng])), wu = __fmul_rn(scu, static_cast<float>(g.rs[nu]));
  const float bg = g.bias ? h2f(g.bias[ng]) : 0.0f, bu = g.bias ? h2f(g.bias[nu]) : 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = 4 * sg + i;
    if (m >= g.M) continue;
    const float ra = __fmul_rn(g.xa[m], 0.0625f);
    const float gv = fp32_result(__fmaf_rn(ra, __fmul_rn(scg, static_cast<float>(accg[i])), __fmaf_rn(g.xb[m], wg, bg)));
    const float uv = fp32_result(__fmaf_rn(ra, __fmul_rn(scu, static_cast<float>(accu[i])), __fmaf_rn(g.xb[m], wu, bu)));
    g.y[m * g.ldy + col] = f2h(fp32_result(swiglu_value(gv, uv)));
  }
}

// ------------------------------------------------------------------ decode-sized kernel
// M <= 16 (token-at-a-time decoding): the GEMM streams the packed weights once from HBM and
// the activations (M x K/2 bytes) stay in L2.  A workgroup owns 16 * NB weight rows (NB
// blocks of 16 output columns; NB is chosen so that there is about one workgroup per CU) and
// its 8 waves split the K range; each wave streams its share of the rows straight into
// registers, SD 64-byte steps ahead.  In a 64-byte step of a row (128 codes) lane
// l = 16 s + r loads the 16 bytes at offset 16 s of activation row r and of weight rows
// n0 + 16 j + r; both operands expand in the same nibble order into two
// v_mfma_i32_16x16x64_i8 k-steps (lane l holds k-slots 16 s .. 16 s + 15 of row r), so the dot
// product is unchanged.  Rows past M or N and bytes past K are out of their buffer ranges and
// read as zeros.  The 8 partial sums are added in LDS; lane n + 16 (m / 4), register m % 4 of
// a block holds D[m][n].
template <int NB, int SD>
struct Skinny {
  static constexpr int WAVES = 8;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int BN = 16 * NB;
  static constexpr int LDS = WAVES * NB * 4 * 64 * 4;  // partial sums: [wave][block][reg][lane] int32
};

// A8: 8-bit activation codes (W4A8): a lane loads the 32 code bytes matching its 32 weight
// codes, in the weights' k-slot order (v_perm_b32) and made signed (xor 0x80, codes - 128);
// the epilogue adds the shift back through the zero-point term (beta + 128 alpha).
template <int NB, int SD, bool A8 = false>
__global__ void __launch_bounds__(512)
w4a4_gemm_skinny(GemmArgs g) {
  using S = Skinny<NB, SD>;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  int* const part = reinterpret_cast<int*>(lds);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15;
  const int sg = lane >> 4;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * S::BN;
  const uint32_t KB = static_cast<uint32_t>(g.K / 2);
  // k range of this wave in bytes, whole 64-byte steps
  const uint32_t kw = ((KB + S::WAVES * 64 - 1) / (S::WAVES * 64)) * 64;
  const uint32_t k0 = wave * kw;
  const int nsteps = static_cast<int>(kw / 64);
  const uint32_t AB = A8 ? 2 * KB : KB;  // activation bytes per row
  const __amdgpu_buffer_rsrc_t rsa = buf_rsrc(g.xq, g.M * AB);
  const __amdgpu_buffer_rsrc_t rsb = buf_rsrc(g.wq, g.N * KB);
  const uint32_t arow = static_cast<uint32_t>(r) * AB;
  uint32_t brow[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) brow[j] = static_cast<uint32_t>(n0 + 16 * j + r) * KB;

  v4u ra[SD], ra2[A8 ? SD : 1], rb[SD][NB];
  auto load = [&](int slot, int t) {
    const uint32_t k = k0 + static_cast<uint32_t>(t) * 64 + 16 * sg;
    const bool ok = k < KB && k < k0 + kw;
    if constexpr (A8) {  // the 32 activation bytes of the lane's 32 weight codes
      ra[slot] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rsa, ok ? arow + 2 * k : 0x80000000u, 0, 0));
      ra2[slot] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rsa, ok ? arow + 2 * k + 16 : 0x80000000u, 0, 0));
    } else {
      ra[slot] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rsa, ok ? arow + k : 0x80000000u, 0, 0));
    }
#pragma unroll
    for (int j = 0; j < NB; ++j)
      rb[slot][j] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rsb, ok ? brow[j] + k : 0x80000000u, 0, 0));
  };
  v4i acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) acc[j] = v4i{0, 0, 0, 0};
  auto step = [&](int slot) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      v4i ea;
      if constexpr (A8) {
        ea = act8_operand(hh == 0 ? ra[slot] : ra2[slot]);
      } else {
        const uint32_t a0 = ra[slot][2 * hh], a1 = ra[slot][2 * hh + 1];
        ea = v4i{static_cast<int>(a0 & 0x0F0F0F0Fu), static_cast<int>((a0 >> 4) & 0x0F0F0F0Fu),
                 static_cast<int>(a1 & 0x0F0F0F0Fu), static_cast<int>((a1 >> 4) & 0x0F0F0F0Fu)};
      }
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const uint32_t b0 = rb[slot][j][2 * hh], b1 = rb[slot][j][2 * hh + 1];
        const v4i eb = {static_cast<int>((b0 << 4) & 0xF0F0F0F0u), static_cast<int>(b0 & 0xF0F0F0F0u),
                        static_cast<int>((b1 << 4) & 0xF0F0F0F0u), static_cast<int>(b1 & 0xF0F0F0F0u)};
        acc[j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ea, eb, acc[j], 0, 0, 0);
      }
    }
  };
#pragma unroll
  for (int d = 0; d < SD; ++d) load(d, d);
  for (int t0 = 0; t0 < nsteps; t0 += SD) {
    static_for<SD>([&](auto dc) {
      constexpr int d = decltype(dc)::value;
      // branch-free: steps past the wave's range are loaded out of range (zeros) and add nothing
      step(d);
      load(d, t0 + d + SD);
    });
  }

  // partial sums of the 8 waves meet in LDS; wave 0 adds them and runs the epilogue
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) part[((wave * NB + j) * 4 + i) * 64 + lane] = acc[j][i];
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w = 1; w < S::WAVES; ++w)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[j][i] += part[((w * NB + j) * 4 + i) * 64 + lane];
  if (!A8 && g.swiglu) {
    // NB % 4 == 0 (n0 % 64 == 0): in each run of four blocks, blocks 0, 1 are gate rows and
    // blocks 2, 3 the up rows of the same 32 output columns, in the same lanes and registers
    if constexpr (NB % 4 == 0) {
#pragma unroll
      for (int jj = 0; jj < NB / 2; ++jj) {
        // gate block j = 4t + s (s = 0, 1) holds output columns n0/2 + 32t + 16s + r
        const int j = 4 * (jj / 2) + (jj % 2);
        decode_store_swiglu(g, acc[j], acc[j + 2], n0 + 16 * j + r, n0 / 2 + 32 * (j / 4) + 16 * (j % 4) + r, sg);
      }
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < NB; ++j) decode_store<A8>(g, acc[j], n0 + 16 * j + r, sg);
}

// Prefetch steps: (NB + 1) 16-byte loads per step.
template <int NB>
constexpr int skinny_depth() {
  return NB <= 4 ? 32 / (NB + 1) : 24 / (NB + 1);
}

template <int NB, int SD, bool A8 = false>
bool fits_skinny(const GemmArgs& g) {
  const int64_t kb = g.K / 2;
  return g.M <= 16 && g.M * kb * (A8 ? 2 : 1) + 64 < (int64_t{1} << 31) &&
         (g.N + 16 * NB) * kb + 64 < (int64_t{1} << 31);
}

template <int NB, int SD, bool A8 = false>
hipError_t launch_skinny(const GemmArgs& g, hipStream_t stream) {
  using S = Skinny<NB, SD>;
  auto kern = w4a4_gemm_skinny<NB, SD, A8>;
  const dim3 grid(static_cast<unsigned>((g.N + S::BN - 1) / S::BN));
  return launch(kern, grid, dim3(S::THREADS), S::LDS, stream, g);
}

// ------------------------------------------------------------------ streaming decode kernel
// 2 < M <= 16 (the dot-product kernel's v_dot8 issue grows with M): the packed weight rows
// stream through LDS by direct copies (buffer_load ... lds) of SEG-byte row segments,
// SEG / 16 lanes per row, so one copy instruction reads 64 / (SEG / 16) rows of SEG
// contiguous bytes (the 16-row kernel's loads take 64 bytes of each of 16 rows).
//   * A workgroup owns nb blocks of 16 weight rows: consecutive ones, or with SW nb / 2 pairs
//     of a gate block and its up block (a finer unit than the groups of four that hold 32
//     output columns: LLaMA-2-70B gate/up has 1792 pairs, 7 per CU, against 896 groups).
//     Its (block, stage) pairs, a stage being SEG bytes of the block's 16 rows, are split
//     evenly over its 8 waves, so where the counts do not divide a wave runs from the end
//     of one block into the next.
//   * Each wave has NS ring slots of its own.  A slot holds the stage's 16 weight rows and
//     the same SEG bytes of activation rows 0-15 (L2-resident), both copied the same way, so
//     the loop's only vector memory operations are copies into LDS: it waits on the wave's
//     own load counter, never on a barrier.  (With the activations loaded into registers
//     the compiler's waits for them held back the copies: 58 against 53 us below.)
//   * In a slot, chunk c (16 bytes) of row r sits at position c ^ r: the copying lane loads
//     the chunk that belongs at its landing position.  The 16 lanes of one LDS read (16 rows,
//     one chunk) then fall on 16 different bank groups.
//   * Lane r + 16 s reads chunk 4 t + s (t < SEG / 64) of weight row r and of activation row
//     r.  Both expand as in the 16-row kernel into two v_mfma_i32_16x16x64_i8 k-steps, so D
//     has that kernel's layout.
//   * A8 (8-bit activation codes, the W4A8 setting, M <= 8): the slot holds activation rows
//     0-7 with the 2 SEG code bytes of the stage's k (32 lanes per row, chunk c of row r at
//     position c ^ r); a lane takes the 32 codes of its weight chunk as two 16-byte reads,
//     made signed and reordered as in the ring kernel (act8_operand), and the epilogue adds
//     the shift back (the 16-row kernel's 8-bit arithmetic).
//   * A wave leaves its sums of every block it touched in LDS; after the loop the waves add
//     the partial sums of a block and apply the 16-row kernel's epilogue (SW: each gate
//     block with its up block), so both kernels give the same bits.
// Measured on MI355X (same data, one process, interleaved, us; against the 16-row kernel):
// LLaMA-2-70B [M x 28672] x [8192 x 28672] 26.2 vs 32.1 (M = 16), 24.3 vs 29.4 (M = 8);
// [M x 8192] x [57344 x 8192] with SiLU 53.1 vs 60.9 (M = 16), 51.4 vs 59.2 (M = 8), in
// groups of four blocks; in pairs 48.2 (M = 16) and 45.8 (M = 8) against 52.5 and 50.9;
// LLaMA-2-7B M = 16: [16 x 11008] x [4096 x 11008] 9.2 vs 11.0, [16 x 4096] x [22016 x 4096]
// with SiLU 15.1 vs 18.1 (pairs: 13.9).
template <int SEG, int NS, bool A8 = false>
struct Stream {
  static constexpr int WAVES = 8;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int LPR = SEG / 16;   // lanes per row in a copy
  static constexpr int RPI = 64 / LPR;   // rows per copy instruction (1 KB)
  static constexpr int CPS = 16 / RPI;   // copies per stage
  static constexpr int XPS = SEG / 64;   // chunks of a row a lane reads per stage
  static constexpr int OPS = 2 * CPS;    // copies per stage: weight rows, then activation rows
  static constexpr int WSTAGE = 16 * SEG;  // the 16 weight rows of a stage
  // then activation rows 0-15 of the same bytes of K; A8: rows 0-7 of 8-bit codes (2 SEG bytes)
  static constexpr int STAGE = 2 * WSTAGE;
  static constexpr int MAXP = 4;         // blocks one wave's run may touch
  static constexpr int RING = WAVES * NS * STAGE;
  static constexpr int LDS = RING + WAVES * MAXP * 1024;
  static_assert(SEG == 256 || SEG == 512, "row segments of 16 or 32 lanes");
  static_assert((NS - 1) * OPS <= 63, "outstanding loads fit the vmcnt counter");
  static_assert(LDS <= 160 * 1024, "LDS of one CU");
};

template <int SEG, int NS, bool SW, bool A8 = false>
__global__ void __launch_bounds__(512)
w4a4_gemm_stream(GemmArgs g, int nb, int spb) {
  using S = Stream<SEG, NS, A8>;
  static_assert(!A8 || (!SW && SEG == 256), "8-bit activations: plain products, 256-byte stages");
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, sg = lane >> 4;
  const uint32_t KB = static_cast<uint32_t>(g.K / 2);
  // Plain: blocks blk0 .. blk0 + nb - 1.  SW: nb / 2 gate/up pairs from pair bx nb / 2 on (the
  // last workgroup may have fewer); pair p is gate block 4 (p / 2) + p % 2 with its up block
  // two further, local blocks 2 i (gate) and 2 i + 1 (up) of pair i.
  const int64_t blk0 = static_cast<int64_t>(blockIdx.x) * nb;
  const int64_t pair0 = static_cast<int64_t>(blockIdx.x) * (nb / 2);
  if constexpr (SW) {
    const int64_t pairs = g.N / 32;
    if (pair0 + nb / 2 > pairs) nb = static_cast<int>(2 * (pairs - pair0));
  }
  auto block_of = [&](int lb) -> int64_t {
    if constexpr (SW) {
      const int64_t pr = pair0 + lb / 2;
      return 4 * (pr / 2) + pr % 2 + 2 * (lb % 2);
    } else {
      return blk0 + lb;
    }
  };
  // offsets are 32-bit: (N + 16 nb) K / 2 < 2^31 is checked on the host; rows past M or N
  // and bytes past K are out of range and read as zeros
  const uint32_t XB = A8 ? 2 * KB : KB;  // activation bytes per row
  const __amdgpu_buffer_rsrc_t rsa = buf_rsrc(g.xq, g.M * XB);
  const __amdgpu_buffer_rsrc_t rsb = buf_rsrc(g.wq, g.N * KB);
  uint8_t* const ring = lds + w * NS * S::STAGE;
  int* const part = reinterpret_cast<int*>(lds + S::RING);  // [wave][MAXP][4][64]
  const int T = nb * spb;
  const int u0 = w * T / S::WAVES, u1 = (w + 1) * T / S::WAVES;  // this wave's (block, stage) run

  // copies: lane i brings row q RPI + i / LPR of the stage, landing at chunk position i % LPR;
  // per lane the row offset and the chunk's byte within the segment are fixed
  const int crow = lane / S::LPR, cpos = lane % S::LPR;
  uint32_t crowk[S::CPS], ccol[S::CPS];
#pragma unroll
  for (int q = 0; q < S::CPS; ++q) {
    const int rr = q * S::RPI + crow;
    crowk[q] = static_cast<uint32_t>(rr) * KB;
    ccol[q] = 16 * static_cast<uint32_t>(cpos ^ rr);
  }
  // A8: an activation copy brings rows 2 q + i / 32 (512 bytes each), landing at chunk
  // position i % 32, which holds chunk (i % 32) ^ row
  const int xrow = lane / 32, xpos = lane % 32;
  uint32_t xrowk[S::CPS], xcol[S::CPS];
#pragma unroll
  for (int q = 0; q < S::CPS; ++q) {
    const int rr = 2 * q + xrow;
    xrowk[q] = static_cast<uint32_t>(rr) * XB;
    xcol[q] = 16 * static_cast<uint32_t>(xpos ^ rr);
  }
  (void)xrowk;
  (void)xcol;
  int ib = u0 / spb, is = u0 - ib * spb, iu = u0;  // the next stage to copy
  // Branch-free: a stage past the run is copied with every byte out of range (zeros).
  auto issue = [&](auto slot_c) {
    constexpr int slot = decltype(slot_c)::value;
    // The slot was read by the previous step: those LDS reads must have returned before the
    // copy is issued (a copy of out-of-range zeros lands almost at once, and the compiler
    // may place the copy right behind the reads).
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt not waited on
    asm volatile("" ::: "memory");
    const uint32_t lim = iu < u1 ? KB : 0u;  // bytes of the row in range
    const uint32_t rbase = static_cast<uint32_t>(block_of(ib) * 16) * KB;
    const uint32_t kst = static_cast<uint32_t>(is) * SEG;
#pragma unroll
    for (int q = 0; q < S::CPS; ++q) {
      const uint32_t k = kst + ccol[q];
      const uint32_t off = k < lim ? rbase + crowk[q] + k : 0x80000000u;
      auto* dst = reinterpret_cast<__attribute__((address_space(3))) void*>(
          reinterpret_cast<uintptr_t>(ring + slot * S::STAGE + q * 1024));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, dst, 16, static_cast<int>(off), 0, 0, 0);
    }
    // activation rows 0-15 of the same bytes, laid out like the weight rows (rows past M
    // are out of range: zeros); A8: rows 0-7, the 2 SEG code bytes of the same k
#pragma unroll
    for (int q = 0; q < S::CPS; ++q) {
      uint32_t off;
      if constexpr (A8) {
        const uint32_t k = 2 * kst + xcol[q];
        off = k < 2 * lim ? xrowk[q] + k : 0x80000000u;
      } else {
        const uint32_t k = kst + ccol[q];
        off = k < lim ? crowk[q] + k : 0x80000000u;
      }
      auto* dst = reinterpret_cast<__attribute__((address_space(3))) void*>(
          reinterpret_cast<uintptr_t>(ring + slot * S::STAGE + S::WSTAGE + q * 1024));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, dst, 16, static_cast<int>(off), 0, 0, 0);
    }
    ++iu;
    if (++is == spb) {
      is = 0;
      ++ib;
    }
  };
  auto flush = [&](const v4i& a, int k) {
#pragma unroll
    for (int i = 0; i < 4; ++i) part[((w * S::MAXP + k) * 4 + i) * 64 + lane] = a[i];
  };

  static_for<NS - 1>([&](auto pc) { issue(pc); });
  v4i acc = {0, 0, 0, 0};
  int cs = u0 - (u0 / spb) * spb;  // stage within its block of the next stage to consume
  int kp = 0;                      // partial-sum slot of the current block
  for (int u = u0; u < u1; u += NS) {
    static_for<NS>([&](auto pc) {
      constexpr int p = decltype(pc)::value;
      issue(std::integral_constant<int, (p + NS - 1) % NS>{});  // stage u + p + NS - 1 (that slot was read last step)
      wait_vm_lgkm0<(NS - 1) * S::OPS>();                         // stage u + p has landed
      asm volatile("" ::: "memory");
      if (u + p < u1) {  // uniform over the wave
        if (cs == spb) {  // the run enters its next block
          flush(acc, kp);
          ++kp;
          acc = v4i{0, 0, 0, 0};
          cs = 0;
        }
        const uint8_t* sb = ring + p * S::STAGE + r * SEG;
#pragma unroll
        for (int t = 0; t < S::XPS; ++t) {
          const int c = 4 * t + sg;  // the lane's chunk of the stage
          const v4u wv = *reinterpret_cast<const v4u*>(sb + 16 * (c ^ r));
          v4u av, av2;
          if constexpr (A8) {  // codes 32 c .. 32 c + 31 of row r (rows past 7: row 0, never stored)
            const int xr = r < 8 ? r : 0;
            const uint8_t* xb = ring + p * S::STAGE + S::WSTAGE + xr * (2 * SEG);
            av = *reinterpret_cast<const v4u*>(xb + 16 * ((2 * c) ^ xr));
            av2 = *reinterpret_cast<const v4u*>(xb + 16 * ((2 * c + 1) ^ xr));
          } else {
            av = *reinterpret_cast<const v4u*>(sb + S::WSTAGE + 16 * (c ^ r));
            av2 = av;
          }
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            v4i ea;
            if constexpr (A8) {
              ea = act8_operand(hh == 0 ? av : av2);
            } else {
              const uint32_t a0 = av[2 * hh], a1 = av[2 * hh + 1];
              ea = v4i{static_cast<int>(a0 & 0x0F0F0F0Fu), static_cast<int>((a0 >> 4) & 0x0F0F0F0Fu),
                       static_cast<int>(a1 & 0x0F0F0F0Fu), static_cast<int>((a1 >> 4) & 0x0F0F0F0Fu)};
            }
            const uint32_t b0 = wv[2 * hh], b1 = wv[2 * hh + 1];
            const v4i eb = {static_cast<int>((b0 << 4) & 0xF0F0F0F0u), static_cast<int>(b0 & 0xF0F0F0F0u),
                            static_cast<int>((b1 << 4) & 0xF0F0F0F0u), static_cast<int>(b1 & 0xF0F0F0F0u)};
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(ea, eb, acc, 0, 0, 0);
          }
        }
        ++cs;
      }
    });
  }
  if (u0 < u1) flush(acc, kp);
  wait_vm_lgkm0<0>();  // copies past the run (zeros) land before the workgroup's LDS is released
  __syncthreads();

  // block b: the partial sums of the waves whose runs meet it, in wave order
  auto block_sum = [&](int b) {
    v4i sum = {0, 0, 0, 0};
#pragma unroll
    for (int v = 0; v < S::WAVES; ++v) {
      const int a0 = v * T / S::WAVES, a1 = (v + 1) * T / S::WAVES;
      if (a0 < a1 && a0 < (b + 1) * spb && a1 > b * spb) {
        const int k = b - a0 / spb;
#pragma unroll
        for (int i = 0; i < 4; ++i) sum[i] += part[((v * S::MAXP + k) * 4 + i) * 64 + lane];
      }
    }
    return sum;
  };
  if constexpr (SW) {  // pair i: gate rows 16 gb + r, output columns 32 (p / 2) + 16 (p % 2) + r
    for (int i = w; i < nb / 2; i += S::WAVES) {
      const int64_t pr = pair0 + i;
      decode_store_swiglu(g, block_sum(2 * i), block_sum(2 * i + 1), block_of(2 * i) * 16 + r,
                          32 * (pr / 2) + 16 * (pr % 2) + r, sg);
    }
  } else {
    for (int b = w; b < nb; b += S::WAVES) decode_store<A8>(g, block_sum(b), (blk0 + b) * 16 + r, sg);
  }
}

// Plans the streaming kernel: about one workgroup per CU (nb blocks of 16 rows each; with
// SiLU nb / 2 gate/up pairs), each wave's run touching at most MAXP blocks.  Returns false
// where it does not apply.
template <int SEG, int NS, bool SW, bool A8 = false>
bool try_stream(const GemmArgs& g, hipStream_t stream, hipError_t* err) {
  using S = Stream<SEG, NS, A8>;
  if (g.M > (A8 ? 8 : 16) || (g.a8 != 0) != A8 || (SW && g.N % 64 != 0)) return false;
  int cus = 0;
  *err = device_cus(&cus);
  if (*err != hipSuccess) return true;
  const int64_t kb = g.K / 2, blocks = (g.N + 15) / 16;
  // plain: blocks in order; SW: gate/up pairs of blocks (N / 32 of them), an even count
  const int64_t units = SW ? g.N / 32 : blocks, per = (units + cus - 1) / cus;
  const int64_t nb = SW ? 2 * per : per;
  const int64_t spb = (kb + SEG - 1) / SEG, T = nb * spb;
  if (nb > 16 || T < S::WAVES || T * S::WAVES >= (int64_t{1} << 31)) return false;
  const int64_t L = (T + S::WAVES - 1) / S::WAVES;  // longest run
  if ((L - 1 + spb - 1) / spb + 1 > S::MAXP) return false;
  if ((g.N + 16 * nb) * kb + 64 >= (int64_t{1} << 31) || g.M * kb * (A8 ? 2 : 1) + 64 >= (int64_t{1} << 31))
    return false;
  constexpr auto kern = w4a4_gemm_stream<SEG, NS, SW, A8>;
  *err = set_max_lds<kern>(S::LDS);
  if (*err != hipSuccess) return true;
  const dim3 grid(static_cast<unsigned>((units + per - 1) / per));
  *err = launch(kern, grid, dim3(S::THREADS), S::LDS, stream, g, static_cast<int>(nb), static_cast<int>(spb));
  return true;
}

// ------------------------------------------------------------------ dot-product decode kernel
// Decode sizes (M <= 2): a few activation rows against the whole weight matrix, a matrix-vector
// product whose cost is reading the packed weights once.  Each wave owns a contiguous run of
// at most 64 output units (a weight row; with SiLU the gate/up row pair of one output column;
// from four activation rows on two neighbouring rows, which then share each activation read)
// and streams the rows of its run whole: in step (u, j) lane l loads the 16 bytes at byte
// 1024 j + 16 l of unit u's row(s), so one load instruction of the wave covers 1 KB of one
// row, and the wave keeps 16 loads in flight.  The activation rows sit in LDS made signed
// (q - 8: every nibble xor 8, rows zero-padded to whole KB); v_dot8_i32_i4 multiplies the
// eight signed 4-bit codes of a weight dword with the eight of the matching activation dword
// (both in the packed nibble order) and adds, so
//   sum_k qa qw = sum_k (qa - 8) qw + 8 rs_n.
// Bytes past K are loaded out of their buffer range and read as zeros.  At the end of a unit
// the wave adds up its 64 lane sums (DPP within rows of 16, permlane swaps across them) and
// lane i keeps unit i; the epilogue runs once per wave, one unit per lane, with the 16-row
// decode kernel's arithmetic (acc16 = 16 acc), so both give the same fp16 results.
// A8 (8-bit activation codes, the W4A8 setting, M <= 2): the LDS rows hold the codes made
// signed (xor 0x80: q - 128) and, in every 8-code group, in the order the weight expansion
// gives (even codes, then odd: v_perm_b32); the weight dword expands to two dwords of 16 x
// code bytes and v_dot4_i32_i8 takes four products at a time, so the unit sums are the 16-row
// kernel's 16 sum (qa - 128) qw and its 8-bit epilogue applies (beta + 128 alpha).
template <int MB, bool SW, bool A8 = false>
struct Gemv {
  static constexpr int WAVES = 8;
  static constexpr int THREADS = 64 * WAVES;
  // weight rows per unit: the gate and up rows of an output column (32 rows apart), or with
  // four and more activation rows two neighbouring rows, which share the activation reads
  static constexpr int RPS = SW || MB >= 4 ? 2 : 1;
  static constexpr int RSTEP = SW ? 32 : 1;  // rows between the rows of a unit
  static constexpr int D = 16 / RPS;         // steps in flight: 16 loads per lane
  static constexpr int RUN = 64;             // units per wave at most
  static constexpr int CH = MB <= 4 ? 4 : 2;  // 8 KB chunks of a 4-bit row: K <= 65536 (32768)
  static constexpr int AB = A8 ? 2 : 1;       // activation bytes per packed weight byte
  static constexpr int MAX_LDS = MB * CH * 8 * 1024 * AB;
  static_assert(!A8 || (!SW && MB <= 2), "8-bit activations: plain products, one or two rows");
};

// sum over the 64 lanes, in every lane
__device__ __forceinline__ int wave_total(int v) {
  v += __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  v += __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  v += __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, false);  // row_half_mirror: the other quad of 8
  v += __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, false);  // row_mirror: the other 8 of 16
  const bool odd_row = (threadIdx.x >> 4) & 1, upper = (threadIdx.x >> 5) & 1;
  const auto s16 = __builtin_amdgcn_permlane16_swap(static_cast<uint32_t>(v), static_cast<uint32_t>(v), false, false);
  v += static_cast<int>(odd_row ? s16[0] : s16[1]);  // the other row of the 32-lane half
  const auto s32 = __builtin_amdgcn_permlane32_swap(static_cast<uint32_t>(v), static_cast<uint32_t>(v), false, false);
  v += static_cast<int>(upper ? s32[0] : s32[1]);    // the other half
  return v;
}

template <int MB, bool SW, bool A8 = false>
__global__ void __launch_bounds__(512)
w4a4_gemv(GemmArgs g) {
  using V = Gemv<MB, SW, A8>;
  constexpr int D = V::D, RPS = V::RPS, RSTEP = V::RSTEP;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t KB = static_cast<uint32_t>(g.K / 2);
  const uint32_t J = (KB + 1023) / 1024;  // 1 KB chunks per row
  const uint32_t AROW = J * 1024 * V::AB;  // LDS bytes per activation row
  // balanced runs: wave w of W owns units [w U / W, (w + 1) U / W)
  const int64_t U = SW ? g.N / 2 : (g.N + RPS - 1) / RPS;
  const int64_t W = static_cast<int64_t>(gridDim.x) * V::WAVES;
  const int64_t gw = static_cast<int64_t>(blockIdx.x) * V::WAVES + wave;
  const int64_t u0 = gw * U / W, u1 = (gw + 1) * U / W;
  const uint32_t run = static_cast<uint32_t>(u1 - u0);
  // weight rows of the run: [row0, rowe); byte offsets are relative to row0
  const int64_t row0 = SW ? 64 * (u0 / 32) : RPS * u0;
  const int64_t rowe = SW ? (u1 > u0 ? 64 * ((u1 + 31) / 32) : row0) : (RPS * u1 < g.N ? RPS * u1 : g.N);
  const __amdgpu_buffer_rsrc_t rsb = buf_rsrc(g.wq + row0 * KB, (rowe - row0) * KB);

  // the epilogue's operands first (lane i: unit i; clamped indices, loaded unconditionally),
  // then the first D steps, then the activations: one round trip for all of them
  const int64_t pe = u0 + (static_cast<uint32_t>(lane) < run ? lane : 0);
  const int64_t ne = pe < U ? (SW ? 64 * (pe / 32) + (pe % 32) : RPS * pe) : 0;  // first row of the unit
  const uint16_t* const bp = g.bias ? g.bias : reinterpret_cast<const uint16_t*>(g.wa);  // no branch around the load
  float esc[RPS];
  int32_t ers[RPS];
  uint16_t eb[RPS];
#pragma unroll
  for (int r = 0; r < RPS; ++r) {
    const int64_t n = ne + RSTEP * r < g.N ? ne + RSTEP * r : g.N - 1;
    esc[r] = g.wa[n];
    ers[r] = g.rs[n];
    eb[r] = bp[n];
  }
  float exa[MB], exb[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) {
    const int64_t mc = m < g.M ? m : g.M - 1;
    exa[m] = g.xa[mc];
    exb[m] = g.xb[mc];
  }

  v4u wb[D][RPS];
  uint32_t lu = 0, lj = 0;  // next step to load: unit lu of the run, chunk lj
  auto load = [&](int slot) {
    const uint32_t k = lj * 1024 + 16 * lane;
    const bool ok = lu < run && k < KB;
    int64_t r;
    if constexpr (SW) {
      const int64_t p = u0 + lu;
      r = 64 * (p / 32) + (p % 32) - row0;  // gate row; the up row is 32 further
    } else {
      r = RPS * lu;  // a second row past N is past the buffer range: zeros
    }
    const uint32_t off = static_cast<uint32_t>(r) * KB + k;
#pragma unroll
    for (int q = 0; q < RPS; ++q)
      wb[slot][q] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rsb, ok ? off + q * RSTEP * KB : 0x80000000u, 0, 0));
    if (++lj == J) {
      lj = 0;
      ++lu;
    }
  };
#pragma unroll
  for (int d = 0; d < D; ++d) load(d);

  // activation rows -> LDS, signed and zero-padded; rows past M are zeros.  A row has at most
  // CH x 8 KB (x 2 with 8-bit codes; fits_gemv); every load is issued before the first
  // write, unconditionally (out of range where there is nothing to load), so that the waits
  // do not serialise them.
  const uint32_t XR = KB * V::AB;  // activation bytes per row in global memory
  const __amdgpu_buffer_rsrc_t rsa = buf_rsrc(g.xq, g.M * XR);
  v4u a[V::CH * V::AB][MB];
#pragma unroll
  for (int h = 0; h < V::CH * V::AB; ++h)
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      const uint32_t o = 16 * (threadIdx.x + h * V::THREADS);
      const bool ok = m < g.M && o < XR;
      a[h][m] = __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(rsa, ok ? m * XR + o : 0x80000000u, 0, 0));
    }
#pragma unroll
  for (int h = 0; h < V::CH * V::AB; ++h)
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      const uint32_t o = 16 * (threadIdx.x + h * V::THREADS);
      const bool ok = m < g.M && o < XR;
      v4u v;
      if constexpr (A8) {  // q - 128, each 8-code group as (even codes | odd codes); bytes past K
                           // meet zero weights
        const v4u d = a[h][m];
        v = v4u{__builtin_amdgcn_perm(d[1], d[0], 0x06040200u), __builtin_amdgcn_perm(d[1], d[0], 0x07050301u),
                __builtin_amdgcn_perm(d[3], d[2], 0x06040200u), __builtin_amdgcn_perm(d[3], d[2], 0x07050301u)} ^
            0x80808080u;
      } else {
        v = a[h][m] ^ (ok ? 0x88888888u : 0u);  // out of range: loaded as zeros
      }
      if (o < AROW) *reinterpret_cast<v4u*>(lds + m * AROW + o) = v;
    }
  __syncthreads();

  int acc[RPS][MB], res[RPS][MB];
#pragma unroll
  for (int r = 0; r < RPS; ++r)
#pragma unroll
    for (int m = 0; m < MB; ++m) acc[r][m] = res[r][m] = 0;
  uint32_t cu = 0, cj = 0;  // step being consumed
  const uint32_t steps = run * J;
  for (uint32_t t0 = 0; t0 < steps; t0 += D) {
    static_for<D>([&](auto dc) {
      constexpr int d = decltype(dc)::value;
      // steps past the run consume zeros (loaded out of range)
      const uint32_t ao = (cj * 1024 + 16 * lane) * V::AB;
#pragma unroll
      for (int m = 0; m < MB; ++m) {
        if constexpr (A8) {  // the lane's 32 codes: 8 dwords, (even | odd) per 8-code group
          const v4u a0 = *reinterpret_cast<const v4u*>(lds + m * AROW + ao);
          const v4u a1 = *reinterpret_cast<const v4u*>(lds + m * AROW + ao + 16);
          const uint32_t av[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t w = wb[d][0][e];
            acc[0][m] = __builtin_amdgcn_sdot4(static_cast<int>(av[2 * e]), static_cast<int>((w << 4) & 0xF0F0F0F0u),
                                               acc[0][m], false);
            acc[0][m] = __builtin_amdgcn_sdot4(static_cast<int>(av[2 * e + 1]), static_cast<int>(w & 0xF0F0F0F0u),
                                               acc[0][m], false);
          }
        } else {
          const v4u a = *reinterpret_cast<const v4u*>(lds + m * AROW + ao);
#pragma unroll
          for (int r = 0; r < RPS; ++r)
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc[r][m] = __builtin_amdgcn_sdot8(static_cast<int>(a[e]), static_cast<int>(wb[d][r][e]), acc[r][m], false);
        }
      }
      load(d);
      if (++cj == J) {
        cj = 0;
        if (cu < run) {  // steps past the run only consumed zeros
#pragma unroll
          for (int r = 0; r < RPS; ++r)
#pragma unroll
            for (int m = 0; m < MB; ++m) {
              const int s = wave_total(acc[r][m]);
              res[r][m] = lane == static_cast<int>(cu) ? s : res[r][m];
              acc[r][m] = 0;
            }
        }
        ++cu;
      }
    });
  }

  if (static_cast<uint32_t>(lane) >= run) return;
  const int64_t p = u0 + lane;
  if constexpr (SW) {
    const float wg = __fmul_rn(esc[0], static_cast<float>(ers[0])), wu = __fmul_rn(esc[1], static_cast<float>(ers[1]));
    const float bg = g.bias ? h2f(eb[0]) : 0.0f, bu = g.bias ? h2f(eb[1]) : 0.0f;
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      if (m >= g.M) break;
      const int ag = (res[0][m] + 8 * ers[0]) * 16, au = (res[1][m] + 8 * ers[1]) * 16;
      const float ra = __fmul_rn(exa[m], 0.0625f);
      const float gv = fp32_result(__fmaf_rn(ra, __fmul_rn(esc[0], static_cast<float>(ag)), __fmaf_rn(exb[m], wg, bg)));
      const float uv = fp32_result(__fmaf_rn(ra, __fmul_rn(esc[1], static_cast<float>(au)), __fmaf_rn(exb[m], wu, bu)));
      g.y[m * g.ldy + p] = f2h(fp32_result(swiglu_value(gv, uv)));
    }
  } else {
#pragma unroll
    for (int r = 0; r < RPS; ++r) {
      const int64_t n = RPS * p + r;
      if (n >= g.N) break;
      const float wn = __fmul_rn(esc[r], static_cast<float>(ers[r]));
      const float bn = g.bias ? h2f(eb[r]) : 0.0f;
#pragma unroll
      for (int m = 0; m < MB; ++m) {
        if (m >= g.M) break;
        // 16 x the sum (A8: 16 x the sum of (qa - 128) qw, with beta + 128 alpha below)
        const int a16 = A8 ? res[r][m] : 16 * (res[r][m] + 8 * ers[r]);
        const float t = __fmul_rn(esc[r], static_cast<float>(a16));
        const float xb = A8 ? __fmaf_rn(128.0f, exa[m], exb[m]) : exb[m];
        const float yv = fp32_result(__fmaf_rn(__fmul_rn(exa[m], 0.0625f), t, __fmaf_rn(xb, wn, bn)));
        g.y[m * g.ldy + n] = f2h(yv);
        if (g.dbg_acc) g.dbg_acc[m * g.N + n] = (a16 >> 4) + (A8 ? 128 * ers[r] : 0);
      }
    }
  }
}

template <int MB, bool SW, bool A8 = false>
bool fits_gemv(const GemmArgs& g) {
  using V = Gemv<MB, SW, A8>;
  const int64_t kb = g.K / 2, lds = MB * ((kb + 1023) / 1024) * 1024 * V::AB;
  return g.M <= MB && lds <= V::MAX_LDS && g.M * kb * V::AB + 64 < (int64_t{1} << 31) && (!SW || g.N % 64 == 0);
}

// About one workgroup of 8 waves per CU, and more where the runs would exceed 64 units.
template <int MB, bool SW, bool A8 = false>
hipError_t launch_gemv(const GemmArgs& g, hipStream_t stream) {
  using V = Gemv<MB, SW, A8>;
  constexpr auto kern = w4a4_gemv<MB, SW, A8>;
  const int lds = static_cast<int>(MB * ((g.K / 2 + 1023) / 1024) * 1024 * V::AB);
  if (lds > 64 * 1024) {
    const hipError_t init = set_max_lds<kern>(V::MAX_LDS);
    if (init != hipSuccess) return init;
  }
  int cus = 0;
  const hipError_t e = device_cus(&cus);
  if (e != hipSuccess) return e;
  const int64_t U = SW ? g.N / 2 : (g.N + V::RPS - 1) / V::RPS;
  int64_t waves = static_cast<int64_t>(cus) * V::WAVES;
  if (waves * V::RUN < U) waves = (U + V::RUN - 1) / V::RUN;
  if (waves > U) waves = U;
  const dim3 grid(static_cast<unsigned>((waves + V::WAVES - 1) / V::WAVES));
  return launch(kern, grid, dim3(V::THREADS), lds, stream, g);
}

// The dot-product kernel for M <= 2 (sets *e and returns true when it covers the
// arguments).  Measured on MI355X against the 16-row decode kernel, same data, interleaved
// (us): LLaMA-2-70B [M x 8192] x [57344 x 8192] with SiLU 41.0 vs 56.6 (M = 1), 42.2 vs
// 56.9 (M = 2); [M x 28672] x [8192 x 28672] 22.9 vs 27.2 (M = 1), 23.7 vs 27.5 (M = 2);
// LLaMA-2-7B [M x 4096] x [22016 x 4096] with SiLU 12.3 vs 16.1 (M = 1), 14.3 vs 16.6
// (M = 2); [M x 11008] x [4096 x 11008] 8.2 vs 8.9 (M = 1).  From three rows the streaming
// kernel is as fast or faster (70B gate/up with SiLU at M = 4 45.1 vs 45.5, down 24.1 vs
// 25.0; [4 x 4096] x [57344 x 4096] with SiLU 25.2 vs 27.2), and with eight rows this
// kernel is bound by its v_dot8 issue.
template <bool SW>
bool try_gemv(const GemmArgs& g, hipStream_t stream, hipError_t* e) {
  if (g.M == 1 && fits_gemv<1, SW>(g)) {
    *e = launch_gemv<1, SW>(g, stream);
    return true;
  }
  if (g.M == 2 && fits_gemv<2, SW>(g)) {
    *e = launch_gemv<2, SW>(g, stream);
    return true;
  }
  return false;
}

// NB = ceil(N / 4096) blocks of 16 rows, about one workgroup per CU of a 256-CU part; from
// NB = 7 on, 8 blocks two steps ahead (measured on MI355X, LLaMA-2-70B: [M x 8192] x
// [57344 x 8192] 58-64 vs 65-72 us, [M x 8192] x [28672 x 8192] 31-36 vs 33-37 us against
// 7 blocks three steps ahead).  Falls back to the register-staged tile kernel when the
// 31-bit buffer offsets do not cover the operands.
hipError_t launch_skinny_sized(const GemmArgs& g, hipStream_t stream);

template <int WM, int WN, int TM, int TN>
hipError_t launch_tile(const GemmArgs& g, hipStream_t stream) {
  constexpr int BM = WM * TM * 32, BN = WN * TN * 32;
  const dim3 grid(static_cast<unsigned>((g.N + BN - 1) / BN), static_cast<unsigned>((g.M + BM - 1) / BM));
  return launch(w4a4_gemm_tile<WM, WN, TM, TN>, grid, dim3(64 * WM * WN), 0, stream, g);
}

template <int NB>
hipError_t try_skinny(const GemmArgs& g, hipStream_t stream) {
  constexpr int SD = skinny_depth<NB>();
  if (fits_skinny<NB, SD>(g)) return launch_skinny<NB, SD>(g, stream);
  return launch_tile<2, 2, 2, 2>(g, stream);
}

hipError_t launch_skinny_sized(const GemmArgs& g, hipStream_t stream) {
  const int64_t nb = (g.N + 4095) / 4096;
  switch (nb <= 1 ? 1 : (nb >= 7 ? 8 : nb)) {
    case 1: return try_skinny<1>(g, stream);
    case 2: return try_skinny<2>(g, stream);
    case 3: return try_skinny<3>(g, stream);
    case 4: return try_skinny<4>(g, stream);
    case 5: return try_skinny<5>(g, stream);
    case 6: return try_skinny<6>(g, stream);
    default: return try_skinny<8>(g, stream);
  }
}

// 8-bit activations take two loads per step: shallower prefetch, at most 4 blocks (8 blocks
// spill at any depth); all three fit without spills.
template <int NB>
hipError_t try_skinny8(const GemmArgs& g, hipStream_t stream) {
  static_assert(NB == 1 || NB == 2 || NB == 4, "A8 decode instantiations");
  constexpr int SD = NB == 1 ? 8 : (NB == 2 ? 6 : 4);
  return fits_skinny<NB, SD, true>(g) ? launch_skinny<NB, SD, true>(g, stream) : hipErrorNotSupported;
}

}  // namespace

// 8-bit activations on the ring, with the W4A4 size classes: at least as many 256 x 256
// tiles as CUs -> 256 x 256 tiles of 8 waves of 64 x 128, three stages (3 x 48 KB of LDS);
// fewer -> 128 x 256 tiles of 8 waves of 64 x 64, four stages.  A wave tile of 64 rows by
// 128 columns reads 8 KB of 8-bit A and 8 KB of packed B from LDS per stage, against 16 and
// 4 KB for 128 x 64 (the W4A4 kernel, whose A is half the bytes, gains nothing from it).
// Measured on MI355X (us, one process, interleaved; 256 x 256 tiles of 64 x 128 vs 128 x 64
// wave tiles): [2048 x 22016 x 4096] 210 vs 229, [4096 x 28672 x 4096] 504 vs 525,
// [4096 x 4096 x 14336] 247 vs 254; and 256 x 256 (128 x 64) vs 128 x 256 tiles:
//   [2048 x 22016 x 4096]   211 vs 255      [4096 x 28672 x 4096]   505 vs 611
//   [4096 x 4096 x 14336]   241 vs 290      [2048 x 4096 x 11008]   150 vs 104 (128 tiles)
// and earlier, 128 x 256 against 128 x 128 (2 per CU, 3 stages) / 256 x 128 (8 waves,
// 3 stages) / 128 x 128 (4 stages) rings and the register-staged tile kernel:
//   [2048 x 22016 x 4096]   290 vs 329 / 315 / 360 / 389
//   [2048 x 4096 x 11008]   118 vs 150 / 131 / 155 / 165
hipError_t launch_w4a8_ring(const GemmArgs& g0, hipStream_t stream) {
  GemmArgs g = g0;
  g.a8 = 1;
  const int64_t tiles256 = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  if (tiles256 >= 256 && fits_ring<4, 2, 2, 4, 3, true>(g)) return launch_ring<4, 2, 2, 4, 3, 1, 1, true>(g, stream);
  if (!fits_ring<2, 4, 2, 2, 4, true>(g)) return hipErrorNotSupported;
  return launch_ring<2, 4, 2, 2, 4, 1, 1, true>(g, stream);
}

hipError_t launch_w4a8_skinny(const GemmArgs& g, hipStream_t stream) {
  if (g.M > 16) return hipErrorNotSupported;
  // one row, or two from 32 MB of weights: the dot-product kernel in its 8-bit mode.
  // Measured on MI355X against the 16-row kernel (us, same data, interleaved): LLaMA-2-70B
  // [M x 8192] x [57344 x 8192] 43.4 vs 71.3 (M = 1), 46.3 vs 73.5 (M = 2); [M x 28672] x
  // [8192 x 28672] 24.3 vs 27.7, 26.8 vs 28.3; LLaMA-2-7B [M x 4096] x [22016 x 4096] 14.9
  // vs 20.2, 17.0 vs 21.1; [M x 11008] x [4096 x 11008] 9.6 vs 9.6, 11.0 vs 9.8.
  if (g.M == 1 && fits_gemv<1, false, true>(g)) return launch_gemv<1, false, true>(g, stream);
  if (g.M == 2 && g.N * (g.K / 2) >= (int64_t{32} << 20) && fits_gemv<2, false, true>(g))
    return launch_gemv<2, false, true>(g, stream);
  // Up to 8 rows: the streaming kernel with 8-bit activation rows, bit-identical to the
  // 16-row kernel (us): LLaMA-2-70B gate+up 47.4 vs 79.5 (M = 8), 44.8 vs 75.8 (M = 3); down
  // 25.9 vs 32.8, 23.9 vs 28.7; LLaMA-2-7B gate+up 13.7 vs 23.8, down 9.6 vs 11.5 (M = 8).
  hipError_t e;
  if (g.M <= 8 && try_stream<256, 2, false, true>(g, stream, &e)) return e;
  const int64_t nb = (g.N + 4095) / 4096;  // the rows-per-workgroup rule of the W4A4 decode kernel
  if (nb <= 1) return try_skinny8<1>(g, stream);
  if (nb <= 3) return try_skinny8<2>(g, stream);
  return try_skinny8<4>(g, stream);
}

hipError_t launch_w4a4_gemm(const GemmArgs& g, hipStream_t stream) {
  if (g.swiglu) {
    // gate/up with SiLU: the ring kernels (block pairs per wave) and the decode kernel with
    // four 16-row blocks (two gate, two up); the same size classes as below
    constexpr int SD4 = skinny_depth<4>(), SD8 = skinny_depth<8>();
    hipError_t e;
    if (try_gemv<true>(g, stream, &e)) return e;
    if (g.M <= 16 && try_stream<256, 2, true>(g, stream, &e)) return e;
    if (g.M <= 16 && g.N > 16384) return fits_skinny<8, SD8>(g) ? launch_skinny<8, SD8>(g, stream) : hipErrorNotSupported;
    if (g.M <= 16) return fits_skinny<4, SD4>(g) ? launch_skinny<4, SD4>(g, stream) : hipErrorNotSupported;
    if (g.M <= 128)
      return fits_ring<2, 2, 2, 2, 4>(g) ? launch_ring<2, 2, 2, 2, 4, 2, 2>(g, stream) : hipErrorNotSupported;
    const int64_t tiles = ((g.M + 255) / 256) * ((g.N + 255) / 256);
    if (tiles >= 256) return fits_ring<2, 4, 4, 2, 4>(g) ? launch_ring<2, 4, 4, 2, 4>(g, stream) : hipErrorNotSupported;
    return fits_ring<2, 2, 4, 2, 3>(g) ? launch_ring<2, 2, 4, 2, 3, 2>(g, stream) : hipErrorNotSupported;
  }
  // Measured on MI355X (LLaMA-2-7B / LLaMA-3-8B MLP shapes, same data, interleaved runs):
  // the 8-wave 256 x 256 ring tile is fastest once there are at least as many of its tiles
  // as CUs (7B gate+up 169 vs 191 us, 8B gate 427 vs 477 us, 8B down 186 vs 212 us); with
  // fewer, 128 x 256 tiles of 8 waves (64 x 64 each) keep every CU busy with two waves per
  // SIMD (7B down 83.5 vs 93.1 us for 256 x 128 tiles of 4 waves, M = 1024: 67.6 vs 77.2
  // us; the gate/up product keeps the 4-wave tiles, 59 vs 61 us at M = 512).  Decode-sized M
  // (<= 16) streams the weights with the skinny kernel (LLaMA-2-70B, M = 16: down
  // [16x28672]x[8192x28672] 31 vs 98 us, gate [16x8192]x[28672x8192] 36 vs 41 us against
  // the tile kernels); 16 < M <= 128 runs 128 x 128 tiles with two K groups per workgroup.
  // Problems whose byte offsets do not fit 31 bits (operands of 2 GB and more) use the
  // register-staged kernel.
  hipError_t e;
  if (try_gemv<false>(g, stream, &e)) return e;
  if (g.M <= 16 && try_stream<256, 2, false>(g, stream, &e)) return e;
  if (g.M <= 16) return launch_skinny_sized(g, stream);
  if (g.M <= 128) {
    if (fits_ring<2, 2, 2, 2, 4>(g)) return launch_ring<2, 2, 2, 2, 4, 2, 2>(g, stream);
    return launch_tile<2, 2, 2, 2>(g, stream);
  }
  const int64_t tiles256 = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  if (tiles256 >= 256) {
    if (fits_ring<2, 4, 4, 2, 4>(g)) return launch_ring<2, 4, 4, 2, 4>(g, stream);
    return launch_tile<2, 4, 4, 2>(g, stream);
  }
  if (fits_ring<2, 4, 2, 2, 3>(g)) return launch_ring<2, 4, 2, 2, 3>(g, stream);
  return launch_tile<2, 4, 4, 2>(g, stream);
}

}  // namespace sq
