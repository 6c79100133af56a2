// Internal declarations shared by the host API and the kernel translation units.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <vector>

namespace sq {

// Host: the library's dense Hadamard factor of order n (1, 28, 172); false if none.
bool hadamard_factor(int n, std::vector<int8_t>* out);

// Arguments of one row-rotation + quantization launch (activations or weights).
struct RotQuantArgs {
  const uint16_t* x;     // fp16 bits [rows, ldx]
  int64_t rows;
  int64_t K;
  int64_t ldx;
  int a;                 // dense factor order
  const int8_t* H;       // [a, a] +-1 (device), nullptr when a == 1
  int b;                 // Sylvester order
  int group;             // quantization group (asym mode)
  int bits;              // activation codes: 4 (two per byte) or 8 (one per byte)
  float clip = 1.0f;     // range clipping ratio in (0, 1] (asym mode; 1 = plain min-max)
  const int8_t* signs = nullptr;  // +-1 [a * b] (device): diagonal S of a random Hadamard S H
  float inv_sqrt_n;      // fl32(1 / sqrt(a * b))
  uint8_t* q;            // codes [rows, K/2] (4-bit, packed) or [rows, K] (8-bit)
  float* alpha;          // [rows, K/group] (asym) or [rows] (sym)
  float* beta;           // [rows, K/group] (asym only)
  int32_t* rowsum;       // [rows] (sym only)
  float* dbg;            // optional fp32 [rows, K]
};

// Rotation + asymmetric per-group 4- or 8-bit quantization of activation rows.
hipError_t launch_had_quant_act(const RotQuantArgs& a, hipStream_t stream);
// Fast path for K = a*b rows with a registered dense order, per-token 4-bit groups;
// hipErrorNotSupported when it does not apply.
hipError_t launch_had_quant_kron(const RotQuantArgs& a, hipStream_t stream);
// Rotation + symmetric per-row 4-bit quantization of weight rows, with code row sums.
hipError_t launch_pack_w4(const RotQuantArgs& a, hipStream_t stream);

struct GemmArgs {
  const uint8_t* xq;
  const float* xa;
  const float* xb;
  int64_t M;
  const uint8_t* wq;
  const float* wa;
  const int32_t* rs;
  int64_t N;
  int64_t K;
  const uint16_t* bias;  // fp16 bits [N] or nullptr
  uint16_t* y;           // fp16 bits [M, ldy]
  int64_t ldy;
  int32_t* dbg_acc;      // optional [M, N]
  int32_t swiglu;        // 1: rows of wq interleave gate and up in blocks of 32 (N % 64 == 0);
                         //    y [M, ldy >= N/2] receives SiLU(gate) * up
  int32_t a8;            // 1: xq holds 8-bit codes [M, K] (set by the W4A8 launchers)
};

// hipErrorNotSupported when no kernel covers the arguments (only with swiglu)
hipError_t launch_w4a4_gemm(const GemmArgs& g, hipStream_t stream);
// The same product with 8-bit activation codes (xq [M, K], one code per byte).
hipError_t launch_w4a8_gemm(const GemmArgs& g, hipStream_t stream);
// Its decode-sized (M <= 16) weight-streaming kernels (the dot-product kernel for one or two
// rows, the LDS-streaming kernel up to 8, the 16-row kernel otherwise); hipErrorNotSupported
// otherwise.
hipError_t launch_w4a8_skinny(const GemmArgs& g, hipStream_t stream);
// Its prefill kernel on the LDS ring of the W4A4 GEMM; hipErrorNotSupported where the 32-bit
// buffer offsets do not cover the operands.
hipError_t launch_w4a8_ring(const GemmArgs& g, hipStream_t stream);

struct AttnArgs {
  const uint16_t* q;     // fp16 [B, H, 128], R3-rotated query of the new token
  const uint8_t* kq;     // [B, S, H, 64] packed 4-bit codes
  const void* ka;        // [B, S, H] group parameters: fp32, or fp16 bits when param16
  const void* kb;
  const uint8_t* vq;
  const void* va;
  const void* vb;
  int param16;
  int64_t B, S, H;       // S * H * 64 < 2^31 (32-bit buffer offsets per head)
  float scale_log2e;     // score scale times log2(e)
  uint16_t* out;         // fp16 [B, H, 128]
  // split over the sequence: chunks of chunk_batches batches of 8 tokens, partial softmax
  // states in part (float [B, H, chunks, kAttnPart]); chunks == 1 needs no part
  int64_t chunks = 1;
  int64_t chunk_batches = 0;
  float* part = nullptr;
};

constexpr int kAttnPart = 132;  // floats per partial state: m, l, 2 unused, 128 dims

// Chunks of the sequence split for a device with `cus` compute units: enough (batch, chunk,
// 16-head group) workgroups of 8 waves to give every CU one, a chunk being whole batches of
// 8 tokens (one per wave), at most 64 chunks (one per lane of the combine).
constexpr int kAttnGroupHeads = 16;  // heads of one workgroup of the split attention (4 lanes each)
constexpr int kAttnSplitWaves = 8;   // its waves, which split the chunk's tokens
constexpr int kAttnBatch = 1;        // tokens of a wave's batch
constexpr int kAttnDepth = 2;        // batches in flight per wave
inline void attn_split(int64_t B, int64_t S, int64_t H, int cus, int64_t& chunks, int64_t& chunk_batches) {
  constexpr int unit = kAttnSplitWaves * kAttnBatch;  // tokens of one batch of the workgroup
  const int64_t nb = (S + unit - 1) / unit;
  const int64_t groups = B * ((H + kAttnGroupHeads - 1) / kAttnGroupHeads);
  int64_t want = groups < cus ? (cus + groups - 1) / groups : 1;
  const int64_t most = nb < 64 ? nb : 64;
  if (want > most) want = most;
  if (want < 1) want = 1;
  chunk_batches = (nb + want - 1) / want;
  chunks = (nb + chunk_batches - 1) / chunk_batches;
}

hipError_t launch_attn_decode_kv4(const AttnArgs& a, hipStream_t stream);
hipError_t launch_attn_decode_split(const AttnArgs& a, hipStream_t stream);

// The library's own scratch for the allocation-free split attention: 8 MiB per device (the
// split of any shape on a device of up to 1000 CUs needs less).
constexpr uint64_t kAttnScratchBytes = uint64_t{8} << 20;
// Device address of that scratch on the current device (looked up once per device).
hipError_t attn_scratch(void** ptr);

struct KvArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  int64_t groups;        // B * S * H (one head vector of D = 128 each)
  float inv_sqrt_d;
  uint16_t* q_rot;
  uint8_t* kq;
  void* ka;              // group parameters: fp32, or fp16 bits when param16
  void* kb;
  uint8_t* vq;
  void* va;
  void* vb;
  float* dbg_k;
  int bits;              // cache codes: 4 (two per byte) or 8 (one per byte)
  float k_clip = 1.0f;   // range clipping ratios of the K and V groups, in (0, 1]
  float v_clip = 1.0f;
  int param16 = 0;       // 1: alpha and beta stored as fp16
};

hipError_t launch_qk_had_kvquant(const KvArgs& a, hipStream_t stream);

// Timing of one entry-point call (armed by sq_time_next_call, per host thread): the start
// event is taken with the first kernel the call launches and the stop event with each
// kernel, so the last one sets it.  Both are null when timing is not armed.
struct LaunchTiming {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
LaunchTiming& launch_timing();

// Raises the dynamic LDS limit of kernel Kern to `bytes`, once per process.  A failed
// attempt is not remembered: the next launch tries again and reports its own status.
template <auto Kern>
hipError_t set_max_lds(int bytes) {
  static std::atomic<bool> done{false};
  if (done.load(std::memory_order_acquire)) return hipSuccess;
  const hipError_t e =
      hipFuncSetAttribute(reinterpret_cast<const void*>(Kern), hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess) done.store(true, std::memory_order_release);
  return e;
}

// Workgroups of kernel Kern (threads, dynamic LDS bytes) that fit one CU, queried once per
// process (after set_max_lds); a failed query is not remembered.
template <auto Kern>
hipError_t blocks_per_cu(int threads, int lds, int* out) {
  static std::atomic<int> cached{0};
  int v = cached.load(std::memory_order_acquire);
  if (v == 0) {
    const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, Kern, threads, lds);
    if (e != hipSuccess) return e;
    if (v < 1) v = 1;
    cached.store(v, std::memory_order_release);
  }
  *out = v;
  return hipSuccess;
}

// Compute units of the current device (queried per device and cached; a failed query is
// not remembered).
inline hipError_t device_cus(int* out) {
  static std::atomic<int> cached[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64) {
    const int v = cached[dev].load(std::memory_order_acquire);
    if (v > 0) {
      *out = v;
      return hipSuccess;
    }
  }
  int n = 0;
  e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  if (n < 1) n = 1;
  if (dev >= 0 && dev < 64) cached[dev].store(n, std::memory_order_release);
  *out = n;
  return hipSuccess;
}

// Every kernel of the library is launched through here.
template <typename... Params, typename... Args>
hipError_t launch(void (*kern)(Params...), dim3 grid, dim3 block, uint32_t lds, hipStream_t stream, Args... args) {
  LaunchTiming& t = launch_timing();
  hipExtLaunchKernelGGL(kern, grid, block, lds, stream, t.start, t.stop, 0, args...);
  t.start = nullptr;  // later kernels of the same call only move the stop event
  return hipGetLastError();
}

}  // namespace sq
