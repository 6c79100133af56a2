// Host side of the C ABI declared in include/sq.h: argument validation, error state
// and kernel launches.  Every check runs before anything is enqueued; on a non-OK
// status nothing is written.
#include "sq.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "sq_internal.h"

namespace {

thread_local std::string g_last_error;
thread_local sq::LaunchTiming g_timing;

// Disarms sq_time_next_call's events when the entry point returns, on every path.
struct TimingScope {
  ~TimingScope() { g_timing = sq::LaunchTiming{}; }
};

sq_status fail(sq_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

sq_status ok() {
  g_last_error.clear();
  return SQ_OK;
}

sq_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(SQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

struct Range {
  const void* p;
  uint64_t bytes;
  const char* name;
};

bool overlap(const Range& a, const Range& b) {
  if (!a.p || !b.p || a.bytes == 0 || b.bytes == 0) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
  return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

// Outputs must not overlap any input or each other.
sq_status check_alias(const std::vector<Range>& ins, const std::vector<Range>& outs) {
  for (size_t i = 0; i < outs.size(); ++i) {
    for (const Range& in : ins)
      if (overlap(outs[i], in)) return fail(SQ_ERR_ALIAS, "output %s overlaps input %s", outs[i].name, in.name);
    for (size_t j = i + 1; j < outs.size(); ++j)
      if (overlap(outs[i], outs[j]))
        return fail(SQ_ERR_ALIAS, "output %s overlaps output %s", outs[i].name, outs[j].name);
  }
  return SQ_OK;
}

// Shared checks of the row-rotation arguments.
sq_status check_rotation(int64_t K, int32_t a, const int8_t* H, int32_t b) {
  if (a < 1 || a > SQ_MAX_DENSE) return fail(SQ_ERR_SHAPE, "had_dense_n=%d outside [1, %d]", a, SQ_MAX_DENSE);
  if ((a == 1) != (H == nullptr))
    return fail(a == 1 ? SQ_ERR_SHAPE : SQ_ERR_NULL, "had_dense must be NULL iff had_dense_n == 1 (n=%d)", a);
  if (!is_pow2(b) || b > 32768) return fail(SQ_ERR_SHAPE, "had_pow2_n=%d is not a power of two in [1, 32768]", b);
  const int64_t n = static_cast<int64_t>(a) * b;
  if (K % n != 0) return fail(SQ_ERR_SHAPE, "rotation width %lld does not divide K=%lld", (long long)n, (long long)K);
  return SQ_OK;
}

sq_status check_rows(int64_t M, int64_t K, int64_t ld, const char* mname) {
  if (M < 0) return fail(SQ_ERR_SHAPE, "%s=%lld < 0", mname, (long long)M);
  if (M > (int64_t{1} << 31) - 1) return fail(SQ_ERR_SHAPE, "%s=%lld too large", mname, (long long)M);
  if (K <= 0 || K > SQ_MAX_ROW) return fail(SQ_ERR_SHAPE, "K=%lld outside (0, %d]", (long long)K, SQ_MAX_ROW);
  if (K % 8 != 0) return fail(SQ_ERR_SHAPE, "K=%lld is not a multiple of 8", (long long)K);
  if (ld < K) return fail(SQ_ERR_SHAPE, "leading dimension %lld < K=%lld", (long long)ld, (long long)K);
  if (ld % 8 != 0) return fail(SQ_ERR_ALIGN, "leading dimension %lld is not a multiple of 8", (long long)ld);
  return SQ_OK;
}

// A range clipping ratio: finite, 0 < r <= 1.
sq_status check_clip(float r, const char* name) {
  if (!(r > 0.0f && r <= 1.0f)) return fail(SQ_ERR_SHAPE, "%s=%g outside (0, 1]", name, static_cast<double>(r));
  return SQ_OK;
}

float inv_sqrt(int64_t n) { return static_cast<float>(1.0 / std::sqrt(static_cast<double>(n))); }

}  // namespace

sq::LaunchTiming& sq::launch_timing() { return g_timing; }

extern "C" {

int32_t sq_abi_version(void) { return SQ_ABI_VERSION; }

const char* sq_last_error(void) { return g_last_error.c_str(); }

sq_status sq_time_next_call(void* start_event, void* stop_event) {
  if (!start_event || !stop_event) return fail(SQ_ERR_NULL, "start_event and stop_event are required");
  g_timing.start = static_cast<hipEvent_t>(start_event);
  g_timing.stop = static_cast<hipEvent_t>(stop_event);
  return ok();
}

sq_status sq_hadamard_factor(int32_t n, int8_t* out_host) {
  if (!out_host) return fail(SQ_ERR_NULL, "out_host is NULL");
  std::vector<int8_t> h;
  if (!sq::hadamard_factor(n, &h)) return fail(SQ_ERR_UNSUPPORTED, "no Hadamard factor of order %d", n);
  std::memcpy(out_host, h.data(), h.size());
  return ok();
}

sq_status sq_had_quant_act_ex(const void* x, int64_t M, int64_t K, int64_t ldx,
                              int32_t had_dense_n, const int8_t* had_dense, int32_t had_pow2_n,
                              const int8_t* signs, int32_t bits, int32_t group, float clip,
                              uint8_t* q_out, float* alpha, float* beta, float* dbg_rot,
                              void* stream) {
  TimingScope timing_scope;
  if (!x || !q_out || !alpha || !beta) return fail(SQ_ERR_NULL, "x, q_out, alpha and beta are required");
  sq_status s = check_rows(M, K, ldx, "M");
  if (s != SQ_OK) return s;
  if ((s = check_rotation(K, had_dense_n, had_dense, had_pow2_n)) != SQ_OK) return s;
  if (bits != 4 && bits != 8) return fail(SQ_ERR_UNSUPPORTED, "bits=%d: 4- and 8-bit activations are implemented", bits);
  if (group <= 0 || group % 2 != 0 || K % group != 0)
    return fail(SQ_ERR_SHAPE, "group=%d must be even and divide K=%lld", group, (long long)K);
  if ((s = check_clip(clip, "clip")) != SQ_OK) return s;
  if (!aligned(x, 16) || !aligned(q_out, 16) || !aligned(alpha, 4) || !aligned(beta, 4) ||
      (dbg_rot && !aligned(dbg_rot, 4)))
    return fail(SQ_ERR_ALIGN, "x and q_out must be 16-byte aligned, scales 4-byte aligned");
  const uint64_t G = static_cast<uint64_t>(K / group);
  const uint64_t um = static_cast<uint64_t>(M);
  const uint64_t xbytes = um ? ((um - 1) * ldx + K) * 2 : 0;
  const uint64_t n = static_cast<uint64_t>(had_dense_n) * had_pow2_n;
  s = check_alias({{x, xbytes, "x"}, {had_dense, static_cast<uint64_t>(had_dense_n) * had_dense_n, "had_dense"},
                   {signs, signs ? n : 0, "signs"}},
                  {{q_out, um * K * bits / 8, "q_out"}, {alpha, um * G * 4, "alpha"}, {beta, um * G * 4, "beta"},
                   {dbg_rot, dbg_rot ? um * K * 4 : 0, "dbg_rot"}});
  if (s != SQ_OK) return s;
  if (M == 0) return ok();
  sq::RotQuantArgs a{};
  a.x = static_cast<const uint16_t*>(x);
  a.rows = M;
  a.K = K;
  a.ldx = ldx;
  a.a = had_dense_n;
  a.H = had_dense;
  a.b = had_pow2_n;
  a.group = group;
  a.bits = bits;
  a.clip = clip;
  a.signs = signs;
  a.inv_sqrt_n = inv_sqrt(static_cast<int64_t>(had_dense_n) * had_pow2_n);
  a.q = q_out;
  a.alpha = alpha;
  a.beta = beta;
  a.dbg = dbg_rot;
  return hip_status(sq::launch_had_quant_act(a, static_cast<hipStream_t>(stream)), "had_quant_act launch");
}

sq_status sq_had_quant_act(const void* x, int64_t M, int64_t K, int64_t ldx,
                           int32_t had_dense_n, const int8_t* had_dense, int32_t had_pow2_n,
                           int32_t bits, int32_t group,
                           uint8_t* q_out, float* alpha, float* beta, float* dbg_rot,
                           void* stream) {
  return sq_had_quant_act_ex(x, M, K, ldx, had_dense_n, had_dense, had_pow2_n, nullptr, bits, group, 1.0f, q_out,
                             alpha, beta, dbg_rot, stream);
}

sq_status sq_pack_w4_ex(const void* w, int64_t N, int64_t K, int64_t ldw,
                        int32_t had_dense_n, const int8_t* had_dense, int32_t had_pow2_n, const int8_t* signs,
                        uint8_t* wq, float* w_alpha, int32_t* w_rowsum, void* stream) {
  TimingScope timing_scope;
  if (!w || !wq || !w_alpha || !w_rowsum) return fail(SQ_ERR_NULL, "w, wq, w_alpha and w_rowsum are required");
  sq_status s = check_rows(N, K, ldw, "N");
  if (s != SQ_OK) return s;
  if ((s = check_rotation(K, had_dense_n, had_dense, had_pow2_n)) != SQ_OK) return s;
  if (!aligned(w, 16) || !aligned(wq, 16) || !aligned(w_alpha, 4) || !aligned(w_rowsum, 4))
    return fail(SQ_ERR_ALIGN, "w and wq must be 16-byte aligned, w_alpha and w_rowsum 4-byte aligned");
  const uint64_t un = static_cast<uint64_t>(N);
  const uint64_t wbytes = un ? ((un - 1) * ldw + K) * 2 : 0;
  const uint64_t n = static_cast<uint64_t>(had_dense_n) * had_pow2_n;
  s = check_alias({{w, wbytes, "w"}, {had_dense, static_cast<uint64_t>(had_dense_n) * had_dense_n, "had_dense"},
                   {signs, signs ? n : 0, "signs"}},
                  {{wq, un * K / 2, "wq"}, {w_alpha, un * 4, "w_alpha"}, {w_rowsum, un * 4, "w_rowsum"}});
  if (s != SQ_OK) return s;
  if (N == 0) return ok();
  sq::RotQuantArgs a{};
  a.x = static_cast<const uint16_t*>(w);
  a.rows = N;
  a.K = K;
  a.ldx = ldw;
  a.a = had_dense_n;
  a.H = had_dense;
  a.b = had_pow2_n;
  a.group = static_cast<int>(K);
  a.clip = 1.0f;
  a.signs = signs;
  a.inv_sqrt_n = inv_sqrt(static_cast<int64_t>(had_dense_n) * had_pow2_n);
  a.q = wq;
  a.alpha = w_alpha;
  a.rowsum = w_rowsum;
  return hip_status(sq::launch_pack_w4(a, static_cast<hipStream_t>(stream)), "pack_w4 launch");
}

sq_status sq_pack_w4(const void* w, int64_t N, int64_t K, int64_t ldw,
                     int32_t had_dense_n, const int8_t* had_dense, int32_t had_pow2_n,
                     uint8_t* wq, float* w_alpha, int32_t* w_rowsum, void* stream) {
  return sq_pack_w4_ex(w, N, K, ldw, had_dense_n, had_dense, had_pow2_n, nullptr, wq, w_alpha, w_rowsum, stream);
}

sq_status sq_w4a4_linear(const uint8_t* xq, const float* x_alpha, const float* x_beta, int64_t M,
                         const uint8_t* wq, const float* w_alpha, const int32_t* w_rowsum,
                         int64_t N, int64_t K, const void* bias, void* y, int64_t ldy,
                         int32_t* dbg_acc, void* stream) {
  TimingScope timing_scope;
  if (!xq || !x_alpha || !x_beta || !wq || !w_alpha || !w_rowsum || !y)
    return fail(SQ_ERR_NULL, "xq, x_alpha, x_beta, wq, w_alpha, w_rowsum and y are required");
  if (M < 0 || M > (int64_t{1} << 31) - 1) return fail(SQ_ERR_SHAPE, "M=%lld out of range", (long long)M);
  if (N <= 0 || N > (int64_t{1} << 31) - 1) return fail(SQ_ERR_SHAPE, "N=%lld out of range", (long long)N);
  if (K <= 0 || K % 64 != 0 || K > (int64_t{1} << 20))
    return fail(SQ_ERR_SHAPE, "K=%lld must be a positive multiple of 64 (and <= 2^20)", (long long)K);
  if (ldy < N) return fail(SQ_ERR_SHAPE, "ldy=%lld < N=%lld", (long long)ldy, (long long)N);
  if (!aligned(xq, 16) || !aligned(wq, 16) || !aligned(y, 2) || !aligned(x_alpha, 4) || !aligned(x_beta, 4) ||
      !aligned(w_alpha, 4) || !aligned(w_rowsum, 4) || (bias && !aligned(bias, 2)) || (dbg_acc && !aligned(dbg_acc, 4)))
    return fail(SQ_ERR_ALIGN, "xq/wq need 16-byte, scales 4-byte and y 2-byte alignment");
  const uint64_t um = static_cast<uint64_t>(M), un = static_cast<uint64_t>(N), uk = static_cast<uint64_t>(K);
  const uint64_t ybytes = um ? ((um - 1) * ldy + un) * 2 : 0;
  sq_status s = check_alias({{xq, um * uk / 2, "xq"}, {x_alpha, um * 4, "x_alpha"}, {x_beta, um * 4, "x_beta"},
                             {wq, un * uk / 2, "wq"}, {w_alpha, un * 4, "w_alpha"}, {w_rowsum, un * 4, "w_rowsum"},
                             {bias, bias ? un * 2 : 0, "bias"}},
                            {{y, ybytes, "y"}, {dbg_acc, dbg_acc ? um * un * 4 : 0, "dbg_acc"}});
  if (s != SQ_OK) return s;
  if (M == 0) return ok();
  sq::GemmArgs g{};
  g.xq = xq;
  g.xa = x_alpha;
  g.xb = x_beta;
  g.M = M;
  g.wq = wq;
  g.wa = w_alpha;
  g.rs = w_rowsum;
  g.N = N;
  g.K = K;
  g.bias = static_cast<const uint16_t*>(bias);
  g.y = static_cast<uint16_t*>(y);
  g.ldy = ldy;
  g.dbg_acc = dbg_acc;
  return hip_status(sq::launch_w4a4_gemm(g, static_cast<hipStream_t>(stream)), "w4a4_linear launch");
}

sq_status sq_w4a8_linear(const uint8_t* xq, const float* x_alpha, const float* x_beta, int64_t M,
                         const uint8_t* wq, const float* w_alpha, const int32_t* w_rowsum,
                         int64_t N, int64_t K, const void* bias, void* y, int64_t ldy,
                         int32_t* dbg_acc, void* stream) {
  TimingScope timing_scope;
  if (!xq || !x_alpha || !x_beta || !wq || !w_alpha || !w_rowsum || !y)
    return fail(SQ_ERR_NULL, "xq, x_alpha, x_beta, wq, w_alpha, w_rowsum and y are required");
  if (M < 0 || M > (int64_t{1} << 31) - 1) return fail(SQ_ERR_SHAPE, "M=%lld out of range", (long long)M);
  if (N <= 0 || N > (int64_t{1} << 31) - 1) return fail(SQ_ERR_SHAPE, "N=%lld out of range", (long long)N);
  if (K <= 0 || K % 64 != 0 || K > (int64_t{1} << 17))
    return fail(SQ_ERR_SHAPE, "K=%lld must be a positive multiple of 64 (and <= 2^17)", (long long)K);
  if (ldy < N) return fail(SQ_ERR_SHAPE, "ldy=%lld < N=%lld", (long long)ldy, (long long)N);
  if (!aligned(xq, 16) || !aligned(wq, 16) || !aligned(y, 2) || !aligned(x_alpha, 4) || !aligned(x_beta, 4) ||
      !aligned(w_alpha, 4) || !aligned(w_rowsum, 4) || (bias && !aligned(bias, 2)) || (dbg_acc && !aligned(dbg_acc, 4)))
    return fail(SQ_ERR_ALIGN, "xq/wq need 16-byte, scales 4-byte and y 2-byte alignment");
  const uint64_t um = static_cast<uint64_t>(M), un = static_cast<uint64_t>(N), uk = static_cast<uint64_t>(K);
  const uint64_t ybytes = um ? ((um - 1) * ldy + un) * 2 : 0;
  sq_status s = check_alias({{xq, um * uk, "xq"}, {x_alpha, um * 4, "x_alpha"}, {x_beta, um * 4, "x_beta"},
                             {wq, un * uk / 2, "wq"}, {w_alpha, un * 4, "w_alpha"}, {w_rowsum, un * 4, "w_rowsum"},
                             {bias, bias ? un * 2 : 0, "bias"}},
                            {{y, ybytes, "y"}, {dbg_acc, dbg_acc ? um * un * 4 : 0, "dbg_acc"}});
  if (s != SQ_OK) return s;
  if (M == 0) return ok();
  sq::GemmArgs g{};
  g.xq = xq;
  g.xa = x_alpha;
  g.xb = x_beta;
  g.M = M;
  g.wq = wq;
  g.wa = w_alpha;
  g.rs = w_rowsum;
  g.N = N;
  g.K = K;
  g.bias = static_cast<const uint16_t*>(bias);
  g.y = static_cast<uint16_t*>(y);
  g.ldy = ldy;
  g.dbg_acc = dbg_acc;
  return hip_status(sq::launch_w4a8_gemm(g, static_cast<hipStream_t>(stream)), "w4a8_linear launch");
}

sq_status sq_w4a4_linear_swiglu(const uint8_t* xq, const float* x_alpha, const float* x_beta, int64_t M,
                                const uint8_t* wq, const float* w_alpha, const int32_t* w_rowsum,
                                int64_t N, int64_t K, const void* bias, void* h, int64_t ldh, void* stream) {
  TimingScope timing_scope;
  if (!xq || !x_alpha || !x_beta || !wq || !w_alpha || !w_rowsum || !h)
    return fail(SQ_ERR_NULL, "xq, x_alpha, x_beta, wq, w_alpha, w_rowsum and h are required");
  if (M < 0 || M > (int64_t{1} << 31) - 1) return fail(SQ_ERR_SHAPE, "M=%lld out of range", (long long)M);
  if (N <= 0 || N % 64 != 0 || N > (int64_t{1} << 31) - 1)
    return fail(SQ_ERR_SHAPE, "N=%lld must be a positive multiple of 64 (gate/up blocks of 32)", (long long)N);
  if (K <= 0 || K % 64 != 0 || K > (int64_t{1} << 20))
    return fail(SQ_ERR_SHAPE, "K=%lld must be a positive multiple of 64 (and <= 2^20)", (long long)K);
  if (ldh < N / 2) return fail(SQ_ERR_SHAPE, "ldh=%lld < N/2=%lld", (long long)ldh, (long long)(N / 2));
  if (!aligned(xq, 16) || !aligned(wq, 16) || !aligned(h, 2) || !aligned(x_alpha, 4) || !aligned(x_beta, 4) ||
      !aligned(w_alpha, 4) || !aligned(w_rowsum, 4) || (bias && !aligned(bias, 2)))
    return fail(SQ_ERR_ALIGN, "xq/wq need 16-byte, scales 4-byte and h 2-byte alignment");
  const uint64_t um = static_cast<uint64_t>(M), un = static_cast<uint64_t>(N), uk = static_cast<uint64_t>(K);
  const uint64_t hbytes = um ? ((um - 1) * ldh + un / 2) * 2 : 0;
  sq_status s = check_alias({{xq, um * uk / 2, "xq"}, {x_alpha, um * 4, "x_alpha"}, {x_beta, um * 4, "x_beta"},
                             {wq, un * uk / 2, "wq"}, {w_alpha, un * 4, "w_alpha"}, {w_rowsum, un * 4, "w_rowsum"},
                             {bias, bias ? un * 2 : 0, "bias"}},
                            {{h, hbytes, "h"}});
  if (s != SQ_OK) return s;
  if (M == 0) return ok();
  sq::GemmArgs g{};
  g.xq = xq;
  g.xa = x_alpha;
  g.xb = x_beta;
  g.M = M;
  g.wq = wq;
  g.wa = w_alpha;
  g.rs = w_rowsum;
  g.N = N;
  g.K = K;
  g.bias = static_cast<const uint16_t*>(bias);
  g.y = static_cast<uint16_t*>(h);
  g.ldy = ldh;
  g.dbg_acc = nullptr;
  g.swiglu = 1;
  const hipError_t e = sq::launch_w4a4_gemm(g, static_cast<hipStream_t>(stream));
  if (e == hipErrorNotSupported)
    return fail(SQ_ERR_UNSUPPORTED, "M=%lld N=%lld K=%lld: byte offsets beyond 31 bits", (long long)M,
                (long long)N, (long long)K);
  return hip_status(e, "w4a4_linear_swiglu launch");
}

sq_status sq_qk_had_kvquant_ex(const void* q, const void* k, const void* v,
                               int64_t B, int64_t S, int64_t H, int64_t D, int32_t bits, int32_t group,
                               float k_clip, float v_clip, int32_t param_bits,
                               void* q_rot, uint8_t* k_q, void* k_alpha, void* k_beta,
                               uint8_t* v_q, void* v_alpha, void* v_beta, float* dbg_k_rot,
                               void* stream) {
  TimingScope timing_scope;
  if (!q || !k || !v || !q_rot || !k_q || !k_alpha || !k_beta || !v_q || !v_alpha || !v_beta)
    return fail(SQ_ERR_NULL, "q, k, v, q_rot, k_q, k_alpha, k_beta, v_q, v_alpha and v_beta are required");
  if (B < 0 || S < 0 || H < 0) return fail(SQ_ERR_SHAPE, "negative B, S or H");
  if (D != 128) return fail(SQ_ERR_UNSUPPORTED, "D=%lld: only head_dim 128 is implemented", (long long)D);
  if (bits != 4 && bits != 8) return fail(SQ_ERR_UNSUPPORTED, "bits=%d: 4- and 8-bit KV are implemented", bits);
  if (group != 128) return fail(SQ_ERR_UNSUPPORTED, "group=%d: only group 128 (= D) is implemented", group);
  sq_status s = check_clip(k_clip, "k_clip");
  if (s != SQ_OK || (s = check_clip(v_clip, "v_clip")) != SQ_OK) return s;
  if (param_bits != 32 && param_bits != 16)
    return fail(SQ_ERR_UNSUPPORTED, "param_bits=%d: fp32 (32) and fp16 (16) group parameters are implemented",
                param_bits);
  const uint64_t groups = static_cast<uint64_t>(B) * static_cast<uint64_t>(S) * static_cast<uint64_t>(H);
  if (groups > (uint64_t{1} << 40)) return fail(SQ_ERR_SHAPE, "B*S*H too large");
  const uint64_t pb = static_cast<uint64_t>(param_bits / 8);  // bytes per group parameter
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(q_rot, 16) || !aligned(k_q, 16) ||
      !aligned(v_q, 16) || !aligned(k_alpha, pb) || !aligned(k_beta, pb) || !aligned(v_alpha, pb) ||
      !aligned(v_beta, pb) || (dbg_k_rot && !aligned(dbg_k_rot, 4)))
    return fail(SQ_ERR_ALIGN, "tensors need 16-byte alignment, group parameters their own size");
  const uint64_t E = groups * 128;
  s = check_alias({{q, E * 2, "q"}, {k, E * 2, "k"}, {v, E * 2, "v"}},
                  {{q_rot, E * 2, "q_rot"}, {k_q, E * bits / 8, "k_q"}, {k_alpha, groups * pb, "k_alpha"},
                   {k_beta, groups * pb, "k_beta"}, {v_q, E * bits / 8, "v_q"}, {v_alpha, groups * pb, "v_alpha"},
                   {v_beta, groups * pb, "v_beta"}, {dbg_k_rot, dbg_k_rot ? E * 4 : 0, "dbg_k_rot"}});
  if (s != SQ_OK) return s;
  if (groups == 0) return ok();
  sq::KvArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.groups = static_cast<int64_t>(groups);
  a.inv_sqrt_d = inv_sqrt(128);
  a.q_rot = static_cast<uint16_t*>(q_rot);
  a.kq = k_q;
  a.ka = k_alpha;
  a.kb = k_beta;
  a.vq = v_q;
  a.va = v_alpha;
  a.vb = v_beta;
  a.dbg_k = dbg_k_rot;
  a.bits = bits;
  a.k_clip = k_clip;
  a.v_clip = v_clip;
  a.param16 = param_bits == 16;
  return hip_status(sq::launch_qk_had_kvquant(a, static_cast<hipStream_t>(stream)), "qk_had_kvquant launch");
}

sq_status sq_qk_had_kvquant(const void* q, const void* k, const void* v,
                            int64_t B, int64_t S, int64_t H, int64_t D, int32_t bits, int32_t group,
                            void* q_rot, uint8_t* k_q, float* k_alpha, float* k_beta,
                            uint8_t* v_q, float* v_alpha, float* v_beta, float* dbg_k_rot,
                            void* stream) {
  return sq_qk_had_kvquant_ex(q, k, v, B, S, H, D, bits, group, 1.0f, 1.0f, 32, q_rot, k_q, k_alpha, k_beta, v_q,
                              v_alpha, v_beta, dbg_k_rot, stream);
}

namespace {

// Validation shared by the decode-attention entry points; fills a (apart from the split).
sq_status attn_args(const void* q_rot, const uint8_t* k_q, const void* k_alpha, const void* k_beta,
                    const uint8_t* v_q, const void* v_alpha, const void* v_beta, int64_t B, int64_t S, int64_t H,
                    int64_t D, float scale, int32_t param_bits, void* out, const void* workspace,
                    uint64_t workspace_bytes, sq::AttnArgs& a) {
  if (!q_rot || !k_q || !k_alpha || !k_beta || !v_q || !v_alpha || !v_beta || !out)
    return fail(SQ_ERR_NULL, "q_rot, k_q, k_alpha, k_beta, v_q, v_alpha, v_beta and out are required");
  if (B < 0 || S < 1 || H < 1) return fail(SQ_ERR_SHAPE, "need B >= 0, S >= 1, H >= 1");
  if (D != 128) return fail(SQ_ERR_UNSUPPORTED, "D=%lld: only head_dim 128 is implemented", (long long)D);
  if (B * H >= (int64_t{1} << 31) || S >= (int64_t{1} << 31) / (H * 64))
    return fail(SQ_ERR_SHAPE, "B*H=%lld or S*H*64 beyond 2^31", (long long)(B * H));
  if (!(std::fabs(scale) < 3.0e38f)) return fail(SQ_ERR_SHAPE, "scale must be finite");
  if (param_bits != 32 && param_bits != 16)
    return fail(SQ_ERR_UNSUPPORTED, "param_bits=%d: fp32 (32) and fp16 (16) group parameters are implemented",
                param_bits);
  const uint64_t pb = static_cast<uint64_t>(param_bits / 8);
  if (!aligned(q_rot, 16) || !aligned(k_q, 16) || !aligned(v_q, 16) || !aligned(out, 16) || !aligned(k_alpha, pb) ||
      !aligned(k_beta, pb) || !aligned(v_alpha, pb) || !aligned(v_beta, pb) || !aligned(workspace, 16))
    return fail(SQ_ERR_ALIGN,
                "q_rot, k_q, v_q, out and the workspace need 16-byte alignment, group parameters their own size");
  const uint64_t heads = static_cast<uint64_t>(B) * static_cast<uint64_t>(H);
  const uint64_t cache = heads * static_cast<uint64_t>(S);
  std::vector<Range> outs = {{out, heads * 256, "out"}};
  if (workspace && workspace_bytes) outs.push_back({workspace, workspace_bytes, "workspace"});
  sq_status s = check_alias({{q_rot, heads * 256, "q_rot"}, {k_q, cache * 64, "k_q"}, {v_q, cache * 64, "v_q"},
                             {k_alpha, cache * pb, "k_alpha"}, {k_beta, cache * pb, "k_beta"},
                             {v_alpha, cache * pb, "v_alpha"}, {v_beta, cache * pb, "v_beta"}},
                            outs);
  if (s != SQ_OK) return s;
  a = sq::AttnArgs{};
  a.q = static_cast<const uint16_t*>(q_rot);
  a.kq = k_q;
  a.ka = k_alpha;
  a.kb = k_beta;
  a.vq = v_q;
  a.va = v_alpha;
  a.vb = v_beta;
  a.B = B;
  a.S = S;
  a.H = H;
  a.scale_log2e = static_cast<float>(static_cast<double>(scale) * 1.4426950408889634);
  a.param16 = param_bits == 16;
  a.out = static_cast<uint16_t*>(out);
  return SQ_OK;
}

// The sequence split on the current device, and the workspace bytes it needs.
sq_status attn_split_here(int64_t B, int64_t S, int64_t H, int64_t& chunks, int64_t& chunk_batches,
                          uint64_t& bytes) {
  int cus = 0;
  const hipError_t e = sq::device_cus(&cus);
  if (e != hipSuccess) return hip_status(e, "compute-unit count of the current device");
  sq::attn_split(B, S, H, cus, chunks, chunk_batches);
  bytes = chunks > 1 ? static_cast<uint64_t>(B) * static_cast<uint64_t>(H) * static_cast<uint64_t>(chunks) *
                           (sq::kAttnPart * 4)
                     : 0;
  return SQ_OK;
}

}  // namespace

sq_status sq_attn_decode_kv4_ex(const void* q_rot, const uint8_t* k_q, const void* k_alpha, const void* k_beta,
                                const uint8_t* v_q, const void* v_alpha, const void* v_beta,
                                int64_t B, int64_t S, int64_t H, int64_t D, float scale, int32_t param_bits,
                                void* out, void* stream) {
  TimingScope timing_scope;
  sq::AttnArgs a;
  const sq_status s = attn_args(q_rot, k_q, k_alpha, k_beta, v_q, v_alpha, v_beta, B, S, H, D, scale, param_bits,
                                out, nullptr, 0, a);
  if (s != SQ_OK) return s;
  if (B == 0) return ok();
  return hip_status(sq::launch_attn_decode_kv4(a, static_cast<hipStream_t>(stream)), "attn_decode_kv4 launch");
}

sq_status sq_attn_decode_workspace(int64_t B, int64_t S, int64_t H, int64_t D, uint64_t* bytes) {
  if (!bytes) return fail(SQ_ERR_NULL, "bytes is required");
  if (B < 0 || S < 1 || H < 1) return fail(SQ_ERR_SHAPE, "need B >= 0, S >= 1, H >= 1");
  if (D != 128) return fail(SQ_ERR_UNSUPPORTED, "D=%lld: only head_dim 128 is implemented", (long long)D);
  if (B * H >= (int64_t{1} << 31) || S >= (int64_t{1} << 31) / (H * 64))
    return fail(SQ_ERR_SHAPE, "B*H=%lld or S*H*64 beyond 2^31", (long long)(B * H));
  int64_t chunks = 1, cb = 0;
  uint64_t need = 0;
  const sq_status s = attn_split_here(B, S, H, chunks, cb, need);
  if (s != SQ_OK) return s;
  *bytes = need;
  return ok();
}

sq_status sq_attn_decode_kv4_split(const void* q_rot, const uint8_t* k_q, const void* k_alpha, const void* k_beta,
                                   const uint8_t* v_q, const void* v_alpha, const void* v_beta,
                                   int64_t B, int64_t S, int64_t H, int64_t D, float scale, int32_t param_bits,
                                   void* out, void* workspace, uint64_t workspace_bytes, void* stream) {
  TimingScope timing_scope;
  sq::AttnArgs a;
  sq_status s = attn_args(q_rot, k_q, k_alpha, k_beta, v_q, v_alpha, v_beta, B, S, H, D, scale, param_bits, out,
                          workspace, workspace_bytes, a);
  if (s != SQ_OK) return s;
  if (B == 0) return ok();
  uint64_t need = 0;
  s = attn_split_here(B, S, H, a.chunks, a.chunk_batches, need);
  if (s != SQ_OK) return s;
  if (workspace_bytes < need || (need > 0 && !workspace))
    return fail(SQ_ERR_SHAPE, "workspace of %llu bytes, %llu needed", (unsigned long long)workspace_bytes,
                (unsigned long long)need);
  a.part = static_cast<float*>(workspace);
  return hip_status(sq::launch_attn_decode_split(a, static_cast<hipStream_t>(stream)), "attn_decode_split launch");
}

sq_status sq_attn_decode_kv4_split_noalloc(const void* q_rot, const uint8_t* k_q, const void* k_alpha,
                                           const void* k_beta, const uint8_t* v_q, const void* v_alpha,
                                           const void* v_beta, int64_t B, int64_t S, int64_t H, int64_t D,
                                           float scale, int32_t param_bits, void* out, void* stream) {
  TimingScope timing_scope;
  sq::AttnArgs a;
  sq_status s = attn_args(q_rot, k_q, k_alpha, k_beta, v_q, v_alpha, v_beta, B, S, H, D, scale, param_bits, out,
                          nullptr, 0, a);
  if (s != SQ_OK) return s;
  if (B == 0) return ok();
  uint64_t need = 0;
  s = attn_split_here(B, S, H, a.chunks, a.chunk_batches, need);
  if (s != SQ_OK) return s;
  if (need > sq::kAttnScratchBytes)
    return fail(SQ_ERR_SHAPE, "the split needs %llu bytes of scratch; this entry point has %llu",
                (unsigned long long)need, (unsigned long long)sq::kAttnScratchBytes);
  void* scratch = nullptr;
  const hipError_t e = sq::attn_scratch(&scratch);
  if (e != hipSuccess) return hip_status(e, "address of the attention scratch");
  a.part = static_cast<float*>(scratch);
  return hip_status(sq::launch_attn_decode_split(a, static_cast<hipStream_t>(stream)), "attn_decode_split launch");
}

sq_status sq_attn_decode_kv4(const void* q_rot, const uint8_t* k_q, const float* k_alpha, const float* k_beta,
                             const uint8_t* v_q, const float* v_alpha, const float* v_beta,
                             int64_t B, int64_t S, int64_t H, int64_t D, float scale, void* out, void* stream) {
  return sq_attn_decode_kv4_ex(q_rot, k_q, k_alpha, k_beta, v_q, v_alpha, v_beta, B, S, H, D, scale, 32, out, stream);
}

}  // extern "C"
