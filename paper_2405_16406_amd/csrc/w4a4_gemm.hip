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
// Prefill kernel (w4a4_gemm_tile): 256 threads per 256 x 128 output tile, 4 waves in a
// 2 x 2 arrangement, each wave a 128 x 64 sub-tile = 4 x 2 MFMA blocks.  K advances in
// stages of 128 (64 packed bytes per row) through a double-buffered packed LDS tile
// (row pitch 72 bytes: a 16-lane group of 8-byte fragment reads hits 16 distinct bank
// pairs); the next stage's global loads are issued before the current stage's MFMAs and
// written to the other buffer afterwards, one barrier per stage.
// Small-M kernel (w4a4_gemm_v1): 128 x 128 tiles, 64-k single-buffered stages; used for
// M < 128.
#include <cstdlib>
#include <utility>

#include "sq_device.h"
#include "sq_internal.h"

namespace sq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

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
  // Tile order.  Consecutive workgroup ids go to different XCDs (round robin over 8), so
  // each XCD is given a contiguous range of tile ids; within it the tile walks M fastest,
  // so the CUs of one XCD share weight (B) tiles in their L2 and each weight tile is read
  // from HBM about once.
  const int tiles_m = gridDim.y;
  const int total = gridDim.x * gridDim.y;
  const int bid = blockIdx.y * gridDim.x + blockIdx.x;
  const int q8 = total / 8, r8 = total % 8;
  const int xcd = bid % 8, idx = bid / 8;
  const int tile = xcd < r8 ? xcd * (q8 + 1) + idx : r8 * (q8 + 1) + (xcd - r8) * q8 + idx;
  const int64_t m0 = static_cast<int64_t>(tile % tiles_m) * BM;
  const int64_t n0 = static_cast<int64_t>(tile / tiles_m) * BN;
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
    const int64_t ka = (kok ? kb : 0) + scol;
    const int64_t kbb = (kb < KB ? kb : 0) + scol;  // B beyond K only meets zeroed A
#pragma unroll
    for (int q = 0; q < kAChunks; ++q) {
      const int64_t r = m0 + srow + q * (THREADS / 4);
      const uint4 v = *reinterpret_cast<const uint4*>(g.xq + (r < ma ? r : ma) * KB + ka);
      ra[q] = kok ? v : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < kBChunks; ++q) {
      const int64_t r = n0 + srow + q * (THREADS / 4);
      rb[q] = *reinterpret_cast<const uint4*>(g.wq + (r < nb ? r : nb) * KB + kbb);
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

  // ---- epilogue: y = (alpha_m s_n) acc + beta_m (s_n rs_n) [+ bias_n], one fma per output.
  // Neighbouring columns sit in neighbouring lanes; even lanes store both as one 32-bit word
  // when the output rows are 4-byte aligned.  One 32 x 32 block at a time (sched_barrier
  // keeps the scheduler from hoisting every block's accumulators at once).
  const bool pair = ((g.ldy & 1) == 0) && ((reinterpret_cast<uintptr_t>(g.y) & 3) == 0) && (g.dbg_acc == nullptr);
  const int c = lane & 31;
  float csn[TN], cwr[TN], cbn[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int64_t n = n0 + wn + j * 32 + c;
    const int64_t nc = n < g.N ? n : g.N - 1;
    csn[j] = g.wa[nc];
    cwr[j] = __fmul_rn(csn[j], static_cast<float>(g.rs[nc]));
    cbn[j] = g.bias ? h2f(g.bias[nc]) : 0.0f;
  }
  static_for<TM>([&](auto ic) {
    constexpr int i = decltype(ic)::value;
    __builtin_amdgcn_sched_barrier(0);
    const int64_t mb = m0 + wm + i * 32 + 4 * (lane >> 5);
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
      const int64_t n = n0 + wn + j * 32 + c;
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

// ------------------------------------------------------------------ int8-LDS tile kernel
// The packed operands are expanded to int8 once per workgroup while staging (instead of
// once per wave per fragment) and the MFMA fragments are read with ds_read_b128.  Rows
// are 128 int8 (one 128-k stage) at a 144-byte LDS pitch, so 16 lanes reading 16 rows hit
// 16 distinct groups of 4 banks.  Global reads are buffer loads: the k advance is an SGPR
// offset and reads past the end of A or B (M and N tails) return zeros.
constexpr int kIPitch = 144;

__device__ __forceinline__ void expand_chunk_act(uint4 d, uint4& lo, uint4& hi) {
  lo = make_uint4(d.x & 0x0F0F0F0Fu, (d.x >> 4) & 0x0F0F0F0Fu, d.y & 0x0F0F0F0Fu, (d.y >> 4) & 0x0F0F0F0Fu);
  hi = make_uint4(d.z & 0x0F0F0F0Fu, (d.z >> 4) & 0x0F0F0F0Fu, d.w & 0x0F0F0F0Fu, (d.w >> 4) & 0x0F0F0F0Fu);
}
__device__ __forceinline__ void expand_chunk_wgt(uint4 d, uint4& lo, uint4& hi) {
  lo = make_uint4((d.x << 4) & 0xF0F0F0F0u, d.x & 0xF0F0F0F0u, (d.y << 4) & 0xF0F0F0F0u, d.y & 0xF0F0F0F0u);
  hi = make_uint4((d.z << 4) & 0xF0F0F0F0u, d.z & 0xF0F0F0F0u, (d.w << 4) & 0xF0F0F0F0u, d.w & 0xF0F0F0F0u);
}

template <int WAVES_M, int WAVES_N, int TM, int TN>
struct I8Tile {
  static constexpr int THREADS = 64 * WAVES_M * WAVES_N;
  static constexpr int BM = WAVES_M * TM * 32;
  static constexpr int BN = WAVES_N * TN * 32;
  static constexpr int STAGE = (BM + BN) * kIPitch;
  static constexpr int LDS = 2 * STAGE;
  static constexpr int ACH = BM * 4 / THREADS;   // packed 16-byte chunks per thread per stage
  static constexpr int BCH = BN * 4 / THREADS;
  static_assert(ACH * THREADS == BM * 4 && BCH * THREADS == BN * 4, "staging split");
};

template <int WAVES_M, int WAVES_N, int TM, int TN, bool KTAIL>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N)
w4a4_gemm_i8lds(GemmArgs g) {
  using T = I8Tile<WAVES_M, WAVES_N, TM, TN>;
  constexpr int BM = T::BM, BN = T::BN, THREADS = T::THREADS;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int tiles_m = gridDim.y;
  const int total = gridDim.x * gridDim.y;
  const int bid = blockIdx.y * gridDim.x + blockIdx.x;
  const int q8 = total / 8, r8 = total % 8;
  const int xcd = bid % 8, idx = bid / 8;
  const int tile = xcd < r8 ? xcd * (q8 + 1) + idx : r8 * (q8 + 1) + (xcd - r8) * q8 + idx;
  const int m0 = (tile % tiles_m) * BM;
  const int n0 = (tile / tiles_m) * BN;
  const int wm = (wave / WAVES_N) * (TM * 32);
  const int wn = (wave % WAVES_N) * (TN * 32);
  const int KB = static_cast<int>(g.K / 2);
  const int nstage = (KB + kBKB - 1) / kBKB;

  const __amdgpu_buffer_rsrc_t ra_rsrc =
      __builtin_amdgcn_make_buffer_rsrc((void*)g.xq, (short)0, static_cast<int>(g.M * KB), 0x00020000);
  const __amdgpu_buffer_rsrc_t rb_rsrc =
      __builtin_amdgcn_make_buffer_rsrc((void*)g.wq, (short)0, static_cast<int>(g.N * KB), 0x00020000);

  // staging: chunk c = tid + q*THREADS covers tile row (c % 16) + 16 (c / 64), packed column (c / 16) % 4
  const int srow = (tid & 15) + 16 * (tid >> 6);
  const int scol = (tid >> 4) & 3;
  const int aoff0 = (m0 + srow) * KB + scol * 16;  // byte offsets of chunk 0; chunk q adds q*THREADS/4 rows
  const int boff0 = (n0 + srow) * KB + scol * 16;
  uint4 pa[T::ACH], pb[T::BCH];
  auto gload = [&](int st) {
    const int kb = st * kBKB;
#pragma unroll
    for (int q = 0; q < T::ACH; ++q)
      pa[q] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                            ra_rsrc, aoff0 + q * (THREADS / 4) * KB, kb, 0));
#pragma unroll
    for (int q = 0; q < T::BCH; ++q)
      pb[q] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                            rb_rsrc, boff0 + q * (THREADS / 4) * KB, kb, 0));
    if constexpr (KTAIL) {
      // a half stage (K % 128 == 64): columns past K belong to the next row; zero A
      const bool z = kb + scol * 16 >= KB;
#pragma unroll
      for (int q = 0; q < T::ACH; ++q) pa[q] = z ? make_uint4(0, 0, 0, 0) : pa[q];
    }
  };
  auto lstore = [&](int buf) {
    uint8_t* base = lds + buf * T::STAGE + srow * kIPitch + scol * 32;
#pragma unroll
    for (int q = 0; q < T::ACH; ++q) {
      uint4 lo, hi;
      expand_chunk_act(pa[q], lo, hi);
      uint8_t* p = base + q * (THREADS / 4) * kIPitch;
      *reinterpret_cast<uint4*>(p) = lo;
      *reinterpret_cast<uint4*>(p + 16) = hi;
    }
#pragma unroll
    for (int q = 0; q < T::BCH; ++q) {
      uint4 lo, hi;
      expand_chunk_wgt(pb[q], lo, hi);
      uint8_t* p = base + (BM + q * (THREADS / 4)) * kIPitch;
      *reinterpret_cast<uint4*>(p) = lo;
      *reinterpret_cast<uint4*>(p + 16) = hi;
    }
  };
  auto read_frags = [&](v4i (&af)[TM], v4i (&bf)[TN], int buf, int ks) {
    const uint8_t* As = lds + buf * T::STAGE + (lane & 31) * kIPitch + ks * 32 + (lane >> 5) * 16;
#pragma unroll
    for (int i = 0; i < TM; ++i) af[i] = *reinterpret_cast<const v4i*>(As + (wm + i * 32) * kIPitch);
#pragma unroll
    for (int j = 0; j < TN; ++j) bf[j] = *reinterpret_cast<const v4i*>(As + (BM + wn + j * 32) * kIPitch);
  };

  v16i acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v16i{};

  gload(0);
  lstore(0);
  __syncthreads();
  v4i af0[TM], bf0[TN], af1[TM], bf1[TN];
  read_frags(af0, bf0, 0, 0);
  auto mfmas = [&](const v4i (&af)[TM], const v4i (&bf)[TN]) {
    static_for<TM>([&](auto ic) {
      static_for<TN>([&](auto jc) {
        constexpr int i = decltype(ic)::value, j = decltype(jc)::value;
        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
      });
    });
  };
  constexpr int NM = TM * TN;
  constexpr int NV = 12 * (T::ACH + T::BCH);  // expansion VALU per thread per stage
  constexpr int NW = 2 * (T::ACH + T::BCH);   // 16-byte LDS stores per thread per stage
  // Every stage is one scheduling region (no branches): the last stage re-reads its own
  // data and stores it into the unused buffer.
  for (int st = 0; st < nstage; ++st) {
    const int buf = st & 1;
    gload(st + 1 < nstage ? st + 1 : st);
    read_frags(af1, bf1, buf, 1);
    mfmas(af0, bf0);
    __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
    read_frags(af0, bf0, buf, 2);
    mfmas(af1, bf1);
    __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
    read_frags(af1, bf1, buf, 3);
    mfmas(af0, bf0);
    __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
    // k-step 3, first half of its MFMAs: interleaved with expanding + storing the next stage
    static_for<TM / 2>([&](auto ic) {
      static_for<TN>([&](auto jc) {
        constexpr int i = decltype(ic)::value, j = decltype(jc)::value;
        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af1[i], bf1[j], acc[i][j], 0, 0, 0);
      });
    });
    lstore(buf ^ 1);
    static_for<NM / 2>([&](auto) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, (2 * NV + NM - 1) / NM, 0);
      __builtin_amdgcn_sched_group_barrier(0x200, (2 * NW + NM - 1) / NM, 0);
    });
    __syncthreads();
    // next stage's first fragments; the second half of k-step 3 covers their latency
    read_frags(af0, bf0, buf ^ 1, 0);
    static_for<TM - TM / 2>([&](auto ic) {
      static_for<TN>([&](auto jc) {
        constexpr int i = TM / 2 + decltype(ic)::value, j = decltype(jc)::value;
        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af1[i], bf1[j], acc[i][j], 0, 0, 0);
      });
    });
    __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, NM - (TM / 2) * TN, 0);
  }

  // ---- epilogue (as in the packed-LDS kernel)
  const bool pair = ((g.ldy & 1) == 0) && ((reinterpret_cast<uintptr_t>(g.y) & 3) == 0) && (g.dbg_acc == nullptr);
  const int c = lane & 31;
  float csn[TN], cwr[TN], cbn[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int64_t n = n0 + wn + j * 32 + c;
    const int64_t nc = n < g.N ? n : g.N - 1;
    csn[j] = g.wa[nc];
    cwr[j] = __fmul_rn(csn[j], static_cast<float>(g.rs[nc]));
    cbn[j] = g.bias ? h2f(g.bias[nc]) : 0.0f;
  }
  static_for<TM>([&](auto ic) {
    constexpr int i = decltype(ic)::value;
    __builtin_amdgcn_sched_barrier(0);
    const int64_t mb = m0 + wm + i * 32 + 4 * (lane >> 5);
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
      const int64_t n = n0 + wn + j * 32 + c;
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

// Buffer offsets are 32-bit: the int8-LDS kernel needs (M + BM) * K/2 and (N + BN) * K/2 below 2^31.
template <int WM, int WN, int TM, int TN>
bool fits_i8(const GemmArgs& g) {
  using T = I8Tile<WM, WN, TM, TN>;
  const int64_t kb = g.K / 2;
  return (g.M + T::BM) * kb < (int64_t{1} << 31) && (g.N + T::BN) * kb < (int64_t{1} << 31);
}

template <int WM, int WN, int TM, int TN, bool KTAIL>
hipError_t launch_i8_t(const GemmArgs& g, hipStream_t stream) {
  using T = I8Tile<WM, WN, TM, TN>;
  auto kern = w4a4_gemm_i8lds<WM, WN, TM, TN, KTAIL>;
  static const hipError_t init = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, T::LDS);
  if (init != hipSuccess) return init;
  const dim3 grid(static_cast<unsigned>((g.N + T::BN - 1) / T::BN), static_cast<unsigned>((g.M + T::BM - 1) / T::BM));
  hipLaunchKernelGGL(kern, grid, dim3(T::THREADS), T::LDS, stream, g);
  return hipGetLastError();
}

template <int WM, int WN, int TM, int TN>
hipError_t launch_i8(const GemmArgs& g, hipStream_t stream) {
  return (g.K % 128) ? launch_i8_t<WM, WN, TM, TN, true>(g, stream) : launch_i8_t<WM, WN, TM, TN, false>(g, stream);
}

// ------------------------------------------------------------------ small-M kernel
constexpr int kSBM = 128;
constexpr int kSBN = 128;
constexpr int kSBKB = 32;
constexpr int kSPitch = 40;

__global__ void __launch_bounds__(256)
w4a4_gemm_v1(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) uint8_t As[kSBM * kSPitch];
  __shared__ __attribute__((aligned(16))) uint8_t Bs[kSBN * kSPitch];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * kSBM;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * kSBN;
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

  const int lr = tid >> 1;
  const int lc = (tid & 1) * 16;
  const int64_t am = m0 + lr;
  const int64_t bn = n0 + lr;
  const uint8_t* arow = g.xq + am * KB + lc;
  const uint8_t* brow = g.wq + bn * KB + lc;
  const bool aok = am < g.M;
  const bool bok = bn < g.N;

  for (int64_t kb = 0; kb < KB; kb += kSBKB) {
    uint4 va = make_uint4(0, 0, 0, 0);
    uint4 vb = make_uint4(0, 0, 0, 0);
    if (aok) va = *reinterpret_cast<const uint4*>(arow + kb);
    if (bok) vb = *reinterpret_cast<const uint4*>(brow + kb);
    __syncthreads();
    *reinterpret_cast<uint2*>(As + lr * kSPitch + lc) = make_uint2(va.x, va.y);
    *reinterpret_cast<uint2*>(As + lr * kSPitch + lc + 8) = make_uint2(va.z, va.w);
    *reinterpret_cast<uint2*>(Bs + lr * kSPitch + lc) = make_uint2(vb.x, vb.y);
    *reinterpret_cast<uint2*>(Bs + lr * kSPitch + lc + 8) = make_uint2(vb.z, vb.w);
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int off = ks * 16 + (lane >> 5) * 8;
      v4i af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = expand_act(*reinterpret_cast<const uint2*>(As + (wm + i * 32 + (lane & 31)) * kSPitch + off));
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bf[j] = expand_wgt(*reinterpret_cast<const uint2*>(Bs + (wn + j * 32 + (lane & 31)) * kSPitch + off));
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
  }
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 2; ++i) store_block(g, acc[i][j], m0 + wm + i * 32, n0 + wn + j * 32 + (lane & 31), lane);
}

template <int WM, int WN, int TM, int TN>
void launch_tile(const GemmArgs& g, hipStream_t stream) {
  constexpr int BM = WM * TM * 32, BN = WN * TN * 32;
  const dim3 grid(static_cast<unsigned>((g.N + BN - 1) / BN), static_cast<unsigned>((g.M + BM - 1) / BM));
  hipLaunchKernelGGL((w4a4_gemm_tile<WM, WN, TM, TN>), grid, dim3(64 * WM * WN), 0, stream, g);
}

}  // namespace

hipError_t launch_w4a4_gemm(const GemmArgs& g, hipStream_t stream) {
  // SQ_GEMM_VARIANT selects a tile shape for tuning experiments (unset: the default).
  const char* env = getenv("SQ_GEMM_VARIANT");
  const int v = env ? atoi(env) : -1;
  switch (v) {
    case 0: launch_tile<2, 2, 4, 2>(g, stream); break;   // 256 x 128, 4 waves of 128 x 64
    case 1: launch_tile<2, 2, 2, 2>(g, stream); break;   // 128 x 128, 4 waves of 64 x 64
    case 2: launch_tile<2, 2, 4, 4>(g, stream); break;   // 256 x 256, 4 waves of 128 x 128
    case 3: launch_tile<2, 1, 4, 4>(g, stream); break;   // 256 x 128, 2 waves of 128 x 128
    case 4: launch_tile<1, 2, 4, 4>(g, stream); break;   // 128 x 256, 2 waves of 128 x 128
    case 5: launch_tile<2, 4, 4, 2>(g, stream); break;   // 256 x 256, 8 waves of 128 x 64
    case 6: if (fits_i8<2, 2, 4, 4>(g)) return launch_i8<2, 2, 4, 4>(g, stream); break;  // 256 x 256, int8 LDS
    case 7: if (fits_i8<2, 2, 4, 2>(g)) return launch_i8<2, 2, 4, 2>(g, stream); break;  // 256 x 128, int8 LDS
    case 8: if (fits_i8<2, 2, 2, 4>(g)) return launch_i8<2, 2, 2, 4>(g, stream); break;  // 128 x 256, int8 LDS
    case 9: {
      const dim3 grid(static_cast<unsigned>((g.N + kSBN - 1) / kSBN), static_cast<unsigned>((g.M + kSBM - 1) / kSBM));
      hipLaunchKernelGGL(w4a4_gemm_v1, grid, dim3(256), 0, stream, g);
      break;
    }
    default: {
      // Measured on MI355X: the 256 x 256 tile (8 waves of 128 x 64) wins once there are
      // enough tiles to fill the 256 CUs; smaller problems use 128 x 128 tiles.
      const int64_t tiles256 = ((g.M + 255) / 256) * ((g.N + 255) / 256);
      if (g.M >= 128 && tiles256 >= 256)
        launch_tile<2, 4, 4, 2>(g, stream);
      else
        launch_tile<2, 2, 2, 2>(g, stream);
      break;
    }
  }
  return hipGetLastError();
}

}  // namespace sq
