/*
 * sq.h -- C ABI of the MI355X (gfx950) rotated W4A4 inference path of SpinQuant
 * (arXiv 2405.16406): online Hadamard rotation + 4-bit activation quantization, offline
 * weight preparation, the int4 x int4 GEMM with its dequantising epilogue, and R3 +
 * 4-bit KV-cache quantization.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers named "device" are HIP device pointers (or memory the device can read
 *    and write).  The caller allocates and owns every buffer, keeps it alive until
 *    the enqueued work has finished, and synchronises.  The library never allocates,
 *    frees or synchronises; it only enqueues kernels on `stream` (a hipStream_t; NULL
 *    means the default stream).  Calls are asynchronous.
 *  - Tensors are row-major.  fp16 is IEEE binary16; scales are fp32.
 *  - 4-bit codes are packed two per byte along the row, the element with the even
 *    index in the low nibble.  Activation and KV codes are unsigned (0..15); weight
 *    codes are two's-complement nibbles (-7..7).
 *  - Quantization follows eq. 1 of the paper (Sec. 2):
 *        X_Q = alpha * round((X - beta) / alpha) + beta,
 *    asymmetric (alpha = (max-min)/(2^N-1), beta = min) for activations and the KV
 *    cache, symmetric (alpha = max|X|/(2^(N-1)-1), beta = 0) for weights, no range
 *    clipping (App. A, "Quantization choice", Table 12).  Round-to-nearest is ties to
 *    even; (X-beta)/alpha is evaluated as (X-beta) * fl32(1/alpha); a group whose
 *    alpha would be zero or subnormal (e.g. a constant group) gets alpha = 1, codes 0.
 *  - Online rotation (R4 on the down-projection input, R3 on Q/K; Sec. 3.1
 *    "Additional unabsorbed rotations"): each contiguous block of n = a*b elements of
 *    a row is multiplied on the right by R = (H_a (x) S_b) / sqrt(n), where H_a is a
 *    +-1 Hadamard matrix of order a and S_b the natural-order Sylvester matrix of order
 *    b = 2^k (dense factor on the outer, strided index: element i = i_a*b + i_b).
 *    (a, b) = (1, 1) is the identity.
 *  - Errors: every argument is checked on the host before anything is enqueued.  A
 *    non-OK status means nothing was enqueued and no output was written; the message
 *    is available from sq_last_error() (per thread).  Launch failures, including "no
 *    device", return SQ_ERR_HIP.  Arguments are never dereferenced on the host.
 */
#ifndef SQ_H_
#define SQ_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SQ_ABI_VERSION 1

/* Largest row length K accepted by sq_had_quant_act / sq_pack_w4 (rotated or not). */
#define SQ_MAX_ROW 32768
/* Largest dense Hadamard factor order a. */
#define SQ_MAX_DENSE 256

typedef enum {
  SQ_OK = 0,
  SQ_ERR_NULL = 1,        /* a required pointer is NULL */
  SQ_ERR_SHAPE = 2,       /* sizes inconsistent or out of range */
  SQ_ERR_UNSUPPORTED = 3, /* a valid request the library does not implement (e.g. bits = 6) */
  SQ_ERR_ALIGN = 4,       /* pointer or leading dimension misaligned */
  SQ_ERR_ALIAS = 5,       /* an output overlaps an input or another output */
  SQ_ERR_HIP = 6          /* the HIP runtime reported an error (no device, launch failure) */
} sq_status;

/* SQ_ABI_VERSION of the built library. */
int32_t sq_abi_version(void);

/* Message for the last non-OK status returned on the calling thread ("" if none). */
const char* sq_last_error(void);

/*
 * sq_time_next_call -- measurement hook, not part of the method.  Arms two events for
 * the next call of sq_had_quant_act(_ex), sq_pack_w4(_ex), sq_w4a4_linear, sq_w4a8_linear,
 * sq_w4a4_linear_swiglu, sq_qk_had_kvquant(_ex) or sq_attn_decode_kv4(_ex)
 * made by this host thread: start_event takes the start time of the first kernel that
 * call launches and stop_event the end time of its last kernel (hipExtLaunchKernel
 * events), so hipEventElapsedTime(start, stop) is the call's time on the device without
 * marker packets between kernels.
 *   start_event, stop_event   hipEvent_t, created by the caller with timing enabled
 * The events are consumed by that next call whatever its outcome; a call that returns
 * an error, or enqueues nothing (M == 0), leaves them as they were.
 * Errors: SQ_ERR_NULL for a NULL event.
 */
sq_status sq_time_next_call(void* start_event, void* stop_event);

/*
 * sq_hadamard_factor -- host helper: writes the library's +-1 Hadamard matrix of order
 * n into out_host[n*n] (row-major int8, HOST memory), for use as `had_dense`.
 *   n = 1    : [1]
 *   n = 28   : Paley type II construction from q = 13
 *   n = 172  : Williamson construction from four symmetric circulants of order 43
 * Any Hadamard matrix is a valid rotation factor (Sec. 3.1 only asks for "a Hadamard
 * matrix"); these are the ones the library provides.  Errors: SQ_ERR_NULL,
 * SQ_ERR_UNSUPPORTED (other n).
 */
sq_status sq_hadamard_factor(int32_t n, int8_t* out_host);

/*
 * sq_had_quant_act -- online Hadamard rotation of every activation row (R4, Sec. 3.1) fused with asymmetric 4-bit quantization of
 * eq. 1 (Sec. 2) and nibble packing, or 8-bit quantization (the W4A8 setting, Sec. 4.2).
 *
 *   x          device fp16 [M, ldx], row stride ldx elements; row m is x[m*ldx .. +K)
 *   M, K       rows (tokens) and row length; M >= 0 (M == 0 is a no-op), 0 < K <= SQ_MAX_ROW,
 *              K % 8 == 0
 *   ldx        >= K, ldx % 8 == 0; x must be 16-byte aligned
 *   had_dense_n  a, order of the dense factor, 1 <= a <= SQ_MAX_DENSE
 *   had_dense  device int8 +-1 [a, a] row-major (must be a Hadamard matrix); NULL iff a == 1
 *   had_pow2_n b, power of two, 1 <= b <= 32768; n = a*b must divide K
 *   bits       4 or 8 (others: SQ_ERR_UNSUPPORTED)
 *   group      quantization group length along the row: group | K, group % 2 == 0;
 *              group == K is per-token quantization (what sq_w4a4_linear consumes)
 *   q_out      device uint8, 16-byte aligned, contiguous: bits 4: [M, K/2] packed codes
 *              0..15 (even k in the low nibble); bits 8: [M, K] codes 0..255
 *   alpha, beta device fp32 [M, K/group] (contiguous): scale and offset of each group
 *   dbg_rot    optional device fp32 [M, K]: the rotated rows (quantizer input); NULL to skip
 *   stream     hipStream_t
 * Errors: SQ_ERR_NULL, SQ_ERR_SHAPE, SQ_ERR_UNSUPPORTED, SQ_ERR_ALIGN, SQ_ERR_ALIAS, SQ_ERR_HIP.
 */
sq_status sq_had_quant_act(const void* x, int64_t M, int64_t K, int64_t ldx,
                           int32_t had_dense_n, const int8_t* had_dense, int32_t had_pow2_n,
                           int32_t bits, int32_t group,
                           uint8_t* q_out, float* alpha, float* beta, float* dbg_rot,
                           void* stream);

/*
 * sq_had_quant_act_ex -- sq_had_quant_act with the two variants the paper compares its
 * choices against (sq_had_quant_act is this call with signs = NULL and clip = 1):
 *   signs      optional device int8 [a*b] (a = had_dense_n, b = had_pow2_n): the diagonal
 *              S of a random Hadamard matrix S H (Sec. 2.2), so that each block of n = a*b
 *              elements is multiplied by S (H_a (x) S_b) / sqrt(n); element i of a block is
 *              multiplied by signs[i] first.  Entries are +1 or -1 (only their sign is read:
 *              negative = -1).  NULL for none.  Any alignment; the matrix-core kernels take
 *              8-byte aligned arrays, others go to the generic kernel.
 *   clip       range clipping ratio r, 0 < r <= 1 (App. A "Quantization choice"): each group
 *              is quantized over [r min, r max] (each end rounded to fp32), so
 *              alpha = fl(fl(r max) - fl(r min)) / L, beta = fl(r min), and codes of values
 *              outside the range clamp to 0 or L.  1 is plain min-max.
 *              Outside (0, 1] (NaN included): SQ_ERR_SHAPE.
 * Every other argument, layout and error as sq_had_quant_act; signs is an input for the
 * overlap check.
 */
sq_status sq_had_quant_act_ex(const void* x, int64_t M, int64_t K, int64_t ldx,
                              int32_t had_dense_n, const int8_t* had_dense, int32_t had_pow2_n,
                              const int8_t* signs, int32_t bits, int32_t group, float clip,
                              uint8_t* q_out, float* alpha, float* beta, float* dbg_rot,
                              void* stream);

/*
 * sq_pack_w4 -- offline weight preparation: optionally absorb the online
 * rotation into the weight, W' = W R (Sec. 3.1: rotations merge into the adjacent
 * weights, so (x R)(W R)^T = x W^T), then symmetric 4-bit quantization of eq. 1 per
 * output channel (row), nibble packing, and the per-row sum of codes used by the
 * epilogue's zero-point term.
 *
 *   w          device fp16 [N, ldw], 16-byte aligned, ldw >= K, ldw % 8 == 0
 *   N, K       output channels and row length; N >= 0, 0 < K <= SQ_MAX_ROW, K % 8 == 0
 *   had_dense_n, had_dense, had_pow2_n   rotation as in sq_had_quant_act ((1, NULL, 1) = none)
 *   wq         device uint8 [N, K/2], 16-byte aligned: two's-complement nibbles -7..7
 *   w_alpha    device fp32 [N]: per-channel scale
 *   w_rowsum   device int32 [N]: sum over k of the codes of row n
 * Errors: as sq_had_quant_act.
 */
sq_status sq_pack_w4(const void* w, int64_t N, int64_t K, int64_t ldw,
                     int32_t had_dense_n, const int8_t* had_dense, int32_t had_pow2_n,
                     uint8_t* wq, float* w_alpha, int32_t* w_rowsum, void* stream);

/*
 * sq_pack_w4_ex -- sq_pack_w4 absorbing the random Hadamard rotation S H of Sec. 2.2:
 * W' = W R with R = S (H_a (x) S_b) / sqrt(n) blockwise, the same R that
 * sq_had_quant_act_ex applies to the activations with the same signs, so that
 * (x R)(W R)^T = x W^T.
 *   signs      optional device int8 [a*b], +1 or -1 (sign read), as in sq_had_quant_act_ex;
 *              NULL makes this call sq_pack_w4
 * Every other argument, layout and error as sq_pack_w4.
 */
sq_status sq_pack_w4_ex(const void* w, int64_t N, int64_t K, int64_t ldw,
                        int32_t had_dense_n, const int8_t* had_dense, int32_t had_pow2_n, const int8_t* signs,
                        uint8_t* wq, float* w_alpha, int32_t* w_rowsum, void* stream);

/*
 * sq_w4a4_linear -- the quantized linear layer y = x W^T on 4-bit codes.  The int4 x int4 products
 * accumulate exactly in int32, acc[m,n] = sum_k qa[m,k] qw[n,k]; the epilogue expands
 * eq. 1 on both operands:
 *     y[m,n] = fp16( w_alpha[n] * (x_alpha[m] * acc[m,n] + x_beta[m] * w_rowsum[n]) + bias[n] )
 *
 *   xq         device uint8 [M, K/2], 16-byte aligned: per-token activation codes
 *              (from sq_had_quant_act with group == K)
 *   x_alpha, x_beta  device fp32 [M]
 *   M          >= 0 (0 is a no-op)
 *   wq, w_alpha, w_rowsum   device, from sq_pack_w4: uint8 [N, K/2] (16-byte aligned), fp32 [N], int32 [N]
 *   N          >= 1
 *   K          > 0, K % 64 == 0, K <= 2^20 (the int32 accumulator holds 16 x acc, and
 *              16 x 15 x 7 x 2^20 < 2^31)
 *   bias       optional device fp16 [N]; NULL for none
 *   y          device fp16 [M, ldy], ldy >= N, 2-byte aligned
 *   dbg_acc    optional device int32 [M, N] (contiguous): the raw accumulators; NULL to skip
 * Errors: SQ_ERR_NULL, SQ_ERR_SHAPE, SQ_ERR_ALIGN, SQ_ERR_ALIAS, SQ_ERR_HIP.
 */
sq_status sq_w4a4_linear(const uint8_t* xq, const float* x_alpha, const float* x_beta, int64_t M,
                         const uint8_t* wq, const float* w_alpha, const int32_t* w_rowsum,
                         int64_t N, int64_t K, const void* bias, void* y, int64_t ldy,
                         int32_t* dbg_acc, void* stream);

/*
 * sq_w4a8_linear -- the quantized linear layer of the W4A8 setting (Sec. 4.2, 4.5): 8-bit
 * per-token activation codes (sq_had_quant_act with bits = 8, group = K) against the 4-bit
 * weights of sq_pack_w4.  acc[m,n] = sum_k qa[m,k] qw[n,k] exactly in int32 and
 *     y[m,n] = fp16( w_alpha[n] * (x_alpha[m] * acc[m,n] + x_beta[m] * w_rowsum[n]) + bias[n] )
 *
 *   xq         device uint8 [M, K] (contiguous), 16-byte aligned: codes 0..255
 *   x_alpha, x_beta, M, wq, w_alpha, w_rowsum, N, bias, y, ldy, dbg_acc   as for sq_w4a4_linear
 *   K          > 0, K % 64 == 0, K <= 2^17 (the int32 sums of 16 x (qa - 128) x qw)
 * Errors: SQ_ERR_NULL, SQ_ERR_SHAPE, SQ_ERR_ALIGN, SQ_ERR_ALIAS, SQ_ERR_HIP.
 */
sq_status sq_w4a8_linear(const uint8_t* xq, const float* x_alpha, const float* x_beta, int64_t M,
                         const uint8_t* wq, const float* w_alpha, const int32_t* w_rowsum,
                         int64_t N, int64_t K, const void* bias, void* y, int64_t ldy,
                         int32_t* dbg_acc, void* stream);

/*
 * sq_w4a4_linear_swiglu -- the gate and up projections of the MLP in one product, combined
 * in the epilogue into the input of down_proj, the activation that R4 rotates (Sec. 3.1,
 * Fig. 1(c)):
 *     h[m,c] = fp16( SiLU(g[m,c]) * u[m,c] ),  SiLU(v) = v / (1 + e^-v),
 * where g and u are the dequantised outputs of sq_w4a4_linear for the gate and up weights,
 * kept in fp32 (not rounded to fp16) before they are combined.
 *
 *   xq, x_alpha, x_beta, M, K, stream   as for sq_w4a4_linear (K <= 2^20)
 *   wq, w_alpha, w_rowsum, bias   the gate and up weights packed by sq_pack_w4 as one
 *              [N, K] matrix whose rows interleave them in blocks of 32: rows 64b .. 64b+31
 *              are gate rows 32b .. 32b+31 and rows 64b+32 .. 64b+63 the up rows of the
 *              same outputs (packing is per row, so this is the two matrices' packed rows
 *              reordered); bias (optional) in the same order
 *   N          2 * I (I outputs), N % 64 == 0
 *   h          device fp16 [M, ldh], ldh >= N/2, 2-byte aligned
 * No raw-accumulator output (sq_w4a4_linear gives the accumulators of the same product).
 * Errors: SQ_ERR_NULL, SQ_ERR_SHAPE, SQ_ERR_ALIGN, SQ_ERR_ALIAS, SQ_ERR_UNSUPPORTED (sizes
 * whose byte offsets exceed 31 bits), SQ_ERR_HIP.
 */
sq_status sq_w4a4_linear_swiglu(const uint8_t* xq, const float* x_alpha, const float* x_beta, int64_t M,
                                const uint8_t* wq, const float* w_alpha, const int32_t* w_rowsum,
                                int64_t N, int64_t K, const void* bias, void* h, int64_t ldh, void* stream);

/*
 * sq_qk_had_kvquant -- R3 (Sec. 3.1) on post-RoPE queries and keys, per head,
 * R = S_D / sqrt(D); then asymmetric 4-bit (or 8-bit: KV8) quantization of eq. 1 of the rotated keys
 * and of the (unrotated) values, one group per `group` contiguous elements of a head
 * vector (group == D: one (alpha, beta) per batch, token and head).
 *
 *   q, k, v    device fp16 [B, S, H, D] contiguous, 16-byte aligned
 *   B, S, H    >= 0 (any zero: no-op); D = 128
 *   bits       4 or 8; group = 128 (= D)
 *   q_rot      device fp16 [B, S, H, D]: Q R, rounded to nearest fp16
 *   k_q, v_q   device uint8, 16-byte aligned: bits 4: [B, S, H, D/2] packed codes 0..15;
 *              bits 8: [B, S, H, D] codes 0..255
 *   k_alpha, k_beta, v_alpha, v_beta   device fp32 [B, S, H, D/group]
 *   dbg_k_rot  optional device fp32 [B, S, H, D]: K R before quantization; NULL to skip
 * Errors: SQ_ERR_NULL, SQ_ERR_SHAPE, SQ_ERR_UNSUPPORTED, SQ_ERR_ALIGN, SQ_ERR_ALIAS, SQ_ERR_HIP.
 */
sq_status sq_qk_had_kvquant(const void* q, const void* k, const void* v,
                            int64_t B, int64_t S, int64_t H, int64_t D, int32_t bits, int32_t group,
                            void* q_rot, uint8_t* k_q, float* k_alpha, float* k_beta,
                            uint8_t* v_q, float* v_alpha, float* v_beta, float* dbg_k_rot,
                            void* stream);

/*
 * sq_qk_had_kvquant_ex -- sq_qk_had_kvquant with range clipping of the cache groups
 * (App. A "Quantization choice" compares clipped and unclipped KV quantizers) and an fp16
 * storage of the group parameters; sq_qk_had_kvquant is this call with k_clip = v_clip = 1
 * and param_bits = 32.
 *   k_clip, v_clip  clipping ratios r, 0 < r <= 1, of the key and value groups: a group is
 *              quantized over [r min, r max] (ends rounded to fp32; for keys the min and max
 *              of the rotated values), codes outside clamp to 0 or L.
 *              Outside (0, 1] (NaN included): SQ_ERR_SHAPE.
 *   param_bits 32: k_alpha, k_beta, v_alpha, v_beta are fp32 [B, S, H, D/group] (4-byte
 *              aligned); 16: fp16 of the same shape (2-byte aligned), half the parameter
 *              bytes of the cache.  fp16 parameters are the fp32 ones rounded to nearest even,
 *              saturated at +-65504; a group whose fp16 alpha is 0 is constant (alpha 1,
 *              codes 0); codes are then taken from the stored pair,
 *              c = clamp(rint((x - beta16) / alpha16), 0, L), each step rounded in fp32.
 *              Other values: SQ_ERR_UNSUPPORTED.
 * Every other argument, layout and error as sq_qk_had_kvquant.
 */
sq_status sq_qk_had_kvquant_ex(const void* q, const void* k, const void* v,
                               int64_t B, int64_t S, int64_t H, int64_t D, int32_t bits, int32_t group,
                               float k_clip, float v_clip, int32_t param_bits,
                               void* q_rot, uint8_t* k_q, void* k_alpha, void* k_beta,
                               uint8_t* v_q, void* v_alpha, void* v_beta, float* dbg_k_rot,
                               void* stream);

/*
 * sq_attn_decode_kv4 -- attention of one new query per (batch, head) over the 4-bit KV
 * cache written by sq_qk_had_kvquant, the step that consumes it.  Keys and values are
 * dequantised group by group with eq. 1, K_t = k_alpha_t * c_t + k_beta_t (in the R3-rotated
 * basis) and V_t likewise; the query is the R3-rotated one (q_rot of sq_qk_had_kvquant), so
 * q_rot . K_t is the score of the unrotated query and key (Sec. 3.1):
 *     out[b,h,:] = fp16( sum_t softmax_t(scale * q_rot[b,h,:] . K_t) V_t ),  t = 0 .. S-1.
 *
 *   q_rot      device fp16 [B, H, 128] (contiguous), 16-byte aligned
 *   k_q, v_q   device uint8 [B, S, H, 64] (the sq_qk_had_kvquant layout), 16-byte aligned
 *   k_alpha, k_beta, v_alpha, v_beta  device fp32 [B, S, H]
 *   B, S, H    B >= 0 (0 is a no-op), S >= 1, H >= 1, B * H < 2^31, S * H * 64 < 2^31
 *   D          128 (others: SQ_ERR_UNSUPPORTED)
 *   scale      finite score scale, e.g. 1/sqrt(128)
 *   out        device fp16 [B, H, 128] (contiguous), 16-byte aligned
 * Errors: SQ_ERR_NULL, SQ_ERR_SHAPE, SQ_ERR_UNSUPPORTED, SQ_ERR_ALIGN, SQ_ERR_ALIAS, SQ_ERR_HIP.
 */
sq_status sq_attn_decode_kv4(const void* q_rot, const uint8_t* k_q, const float* k_alpha, const float* k_beta,
                             const uint8_t* v_q, const float* v_alpha, const float* v_beta,
                             int64_t B, int64_t S, int64_t H, int64_t D, float scale, void* out, void* stream);

/*
 * sq_attn_decode_kv4_ex -- sq_attn_decode_kv4 over a cache whose group parameters are stored
 * as written by sq_qk_had_kvquant_ex with the same param_bits (32: fp32, 16: fp16 [B, S, H],
 * aligned to their size); sq_attn_decode_kv4 is this call with param_bits = 32.
 * Other param_bits: SQ_ERR_UNSUPPORTED.  Every other argument, layout and error as
 * sq_attn_decode_kv4.
 */
sq_status sq_attn_decode_kv4_ex(const void* q_rot, const uint8_t* k_q, const void* k_alpha, const void* k_beta,
                                const uint8_t* v_q, const void* v_alpha, const void* v_beta,
                                int64_t B, int64_t S, int64_t H, int64_t D, float scale, int32_t param_bits,
                                void* out, void* stream);

/*
 * sq_attn_decode_workspace -- device bytes of the workspace sq_attn_decode_kv4_split needs
 * for B, S, H and D on the CURRENT device (the split depends on its compute-unit count):
 * B * H * chunks * 528, where chunks is the number of pieces the S tokens are split into
 * (0 bytes when they are not split).  Shape rules and errors of sq_attn_decode_kv4;
 * SQ_ERR_NULL for a NULL bytes; SQ_ERR_HIP when the device cannot be queried.
 */
sq_status sq_attn_decode_workspace(int64_t B, int64_t S, int64_t H, int64_t D, uint64_t* bytes);

/*
 * sq_attn_decode_kv4_split -- the attention of sq_attn_decode_kv4_ex (same formula, Sec. 3.1
 * R3 with eq. 1 dequantisation), split over the sequence as in flash-decoding: each
 * workgroup reads one chunk of tokens for 16 heads at once, 1 KB of one token per wave
 * load; a second kernel merges the chunks' partial softmax states (maximum, sum,
 * 128 weighted dims, in fp32) in chunk order.  The result equals sq_attn_decode_kv4_ex's
 * up to the order of fp32 additions, and is deterministic.
 *   workspace        device memory, 16-byte aligned, at least the bytes
 *                    sq_attn_decode_workspace gives (NULL allowed when that is 0); the
 *                    caller owns it; its contents need no initialisation and are scratch
 *                    after the call; it must not overlap any argument
 *   workspace_bytes  its size in bytes
 * Every other argument, layout and error as sq_attn_decode_kv4_ex; SQ_ERR_SHAPE when the
 * workspace is too small, SQ_ERR_ALIGN / SQ_ERR_ALIAS for its alignment and overlaps.
 * Calls that share a workspace must be ordered (same stream, or synchronised).
 */
sq_status sq_attn_decode_kv4_split(const void* q_rot, const uint8_t* k_q, const void* k_alpha, const void* k_beta,
                                   const uint8_t* v_q, const void* v_alpha, const void* v_beta,
                                   int64_t B, int64_t S, int64_t H, int64_t D, float scale, int32_t param_bits,
                                   void* out, void* workspace, uint64_t workspace_bytes, void* stream);

/*
 * sq_attn_decode_kv4_split_noalloc -- sq_attn_decode_kv4_split for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid it): the same kernels, with the partial states in the library's own scratch, a
 * file-scope device array of 8 MiB per GPU, held from its first use until the process
 * ends.  The call allocates nothing and frees nothing.
 * The scratch is shared by every call on the same GPU and keeps the last call's contents
 * (no part of it needs clearing: a call writes every state it reads).  Calls that overlap
 * on one GPU race: order them (same stream, or synchronised).
 * Arguments, layouts and errors as sq_attn_decode_kv4_split without the workspace;
 * SQ_ERR_SHAPE when the split needs more than the 8 MiB (sq_attn_decode_workspace gives
 * the bytes; on MI355X no valid shape needs more than about 4.3 MiB).
 */
sq_status sq_attn_decode_kv4_split_noalloc(const void* q_rot, const uint8_t* k_q, const void* k_alpha,
                                           const void* k_beta, const uint8_t* v_q, const void* v_alpha,
                                           const void* v_beta, int64_t B, int64_t S, int64_t H, int64_t D,
                                           float scale, int32_t param_bits, void* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SQ_H_ */
