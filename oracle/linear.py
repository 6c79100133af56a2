"""The rotated W4A4 linear layer of SpinQuant_had (Sec. 3.1; Fig. 1(c)), step by step.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Forward of one quantized linear layer y = x W^T with an online rotation R in front:
  1. had_quant_act: y_rot = x R (rotate.rotate_rows), then per-token asymmetric
     quantization of eq. 1 (granularity per token: Sec. 2 Fig. 2 caption; asymmetric,
     unclipped: App. A Table 12) and nibble packing.
  2. pack_w4 (offline): the rotation is absorbed into the weight (Sec. 3.1: rotations
     merge into the adjacent weights), W' = W R, so (x R)(W R)^T = x W^T; then
     symmetric per-output-channel quantization of eq. 1 and packing.  The per-row sum
     of weight codes is kept for the zero-point term of the epilogue.
  3. gemm_exact: acc[m, n] = sum_k qa[m, k] qw[n, k], exact integers.
  4. epilogue: dequantising eq. 1 on both sides gives
         y[m, n] = sum_k (alpha_m qa[m,k] + beta_m) (s_n qw[n,k])
                 = s_n (alpha_m acc[m, n] + beta_m rowsum[n])
     computed in fp64 and rounded once to fp16.
  5. swiglu_linear: the gate and up projections of the same input combined as
     SiLU(gate) * up (the input of down_proj, which R4 rotates), rounded once to fp16.
"""

import numpy as np

from .quant import pack_nibbles, quant_asym, quant_sym, store_codes
from .rotate import rotate_rows


def _signed(x: np.ndarray, signs, n: int) -> np.ndarray:
    """x with element i multiplied by signs[i % n]: the diagonal S of a random Hadamard
    matrix S H (Sec. 2.2 footnote) applied to every rotation block; exact in fp64."""
    x64 = np.asarray(x, dtype=np.float64)
    if signs is None:
        return x64
    s = np.asarray(signs, dtype=np.float64)
    return x64 * np.tile(s, x64.shape[-1] // n)


def had_quant_act(x: np.ndarray, had_dense, pow2_n: int, bits: int = 4, group: int | None = None,
                  clip: float = 1.0, signs=None):
    """Rotate each row of x (fp16 [M, K]) and quantize it asymmetrically per group.

    had_dense: int8 +-1 [a, a] or None (a = 1); pow2_n = b; rotation block n = a*b.
    (had_dense None, pow2_n 1) is the identity.  clip < 1 clips the range (quant_asym);
    signs (+-1 [a * pow2_n] or None) make the rotation S (H_a (x) S_b) / sqrt(n), a random
    Hadamard matrix.  Returns
    (packed uint8 [M, K/2] (bits 4) or [M, K] (bits 8), alpha fp32 [M, K/group],
     beta fp32 [M, K/group], y_rot fp32 [M, K] = the quantizer input, codes int64 [M, K]).
    """
    x = np.asarray(x)
    a = 1 if had_dense is None else had_dense.shape[0]
    if a * pow2_n == 1 and signs is None:
        y32 = x.astype(np.float32)
    else:
        y32 = rotate_rows(_signed(x, signs, a * pow2_n), had_dense, pow2_n).astype(np.float32)
    q, alpha, beta = quant_asym(y32, bits=bits, group=group, clip=clip)
    return store_codes(q, bits), alpha, beta, y32, q


def pack_w4(w: np.ndarray, had_dense=None, pow2_n: int = 1, bits: int = 4, signs=None):
    """Offline weight preparation: W' = W R (optional), per-row symmetric quant, pack.

    w: fp16 [N, K].  signs as in had_quant_act (the same R folded into the weights).
    Returns (packed uint8 [N, K/2], alpha fp32 [N], rowsum int32 [N], codes int64 [N, K]).
    """
    w = np.asarray(w)
    a = 1 if had_dense is None else had_dense.shape[0]
    if a * pow2_n == 1 and signs is None:
        w32 = w.astype(np.float32)
    else:
        w32 = rotate_rows(_signed(w, signs, a * pow2_n), had_dense, pow2_n).astype(np.float32)
    q, alpha = quant_sym(w32, bits=bits)
    rowsum = q.sum(axis=-1).astype(np.int32)
    return pack_nibbles(q), alpha[..., 0], rowsum, q


def gemm_exact(qa: np.ndarray, qw: np.ndarray) -> np.ndarray:
    """acc = qa qw^T exactly, as int64.

    Computed with an fp64 matrix product: every operand and every partial sum is an
    integer of magnitude below 2^53, so each fp64 operation is exact whatever the
    summation order, and the result equals the integer product.
    """
    qa64 = np.asarray(qa, dtype=np.float64)
    qw64 = np.asarray(qw, dtype=np.float64)
    bound = np.abs(qa64).max(initial=0) * np.abs(qw64).max(initial=0) * qa64.shape[-1]
    if bound >= 2.0 ** 53:
        raise ValueError("integer GEMM would not be exact in fp64")
    return np.rint(qa64 @ qw64.T).astype(np.int64)


def epilogue_f64(acc: np.ndarray, a_alpha: np.ndarray, a_beta: np.ndarray, w_alpha: np.ndarray,
                 w_rowsum: np.ndarray, bias: np.ndarray | None = None) -> np.ndarray:
    """s_n (alpha_m acc + beta_m rowsum_n) [+ bias_n] in fp64, before the output rounding."""
    acc64 = np.asarray(acc, dtype=np.float64)
    am = np.asarray(a_alpha, dtype=np.float64).reshape(-1, 1)
    bm = np.asarray(a_beta, dtype=np.float64).reshape(-1, 1)
    sn = np.asarray(w_alpha, dtype=np.float64).reshape(1, -1)
    rs = np.asarray(w_rowsum, dtype=np.float64).reshape(1, -1)
    y = sn * (am * acc64 + bm * rs)
    if bias is not None:
        y = y + np.asarray(bias, dtype=np.float64).reshape(1, -1)
    return y


def epilogue(acc: np.ndarray, a_alpha: np.ndarray, a_beta: np.ndarray, w_alpha: np.ndarray,
             w_rowsum: np.ndarray, bias: np.ndarray | None = None) -> np.ndarray:
    """y = fp16( s_n (alpha_m acc + beta_m rowsum_n) [+ bias_n] ), fp64 then one rounding."""
    return epilogue_f64(acc, a_alpha, a_beta, w_alpha, w_rowsum, bias).astype(np.float16)


def w4a4_linear(qa, a_alpha, a_beta, qw, w_alpha, w_rowsum, bias=None):
    """GEMM + epilogue on unpacked codes.  Returns (y fp16 [M, N], acc int64 [M, N])."""
    acc = gemm_exact(qa, qw)
    return epilogue(acc, a_alpha, a_beta, w_alpha, w_rowsum, bias), acc


def silu(v: np.ndarray) -> np.ndarray:
    """SiLU(v) = v / (1 + e^-v) in fp64 (the gate activation of the LLaMA MLP)."""
    v = np.asarray(v, dtype=np.float64)
    with np.errstate(over="ignore"):
        return v / (1.0 + np.exp(-v))


def swiglu_linear(qa, a_alpha, a_beta, qw_gate, wa_gate, rs_gate, qw_up, wa_up, rs_up,
                  bias_gate=None, bias_up=None):
    """Gate and up projections of the MLP whose product feeds down_proj (Fig. 1(c): R4 sits
    on that input), h = fp16( SiLU(g) * u ).

    g and u are the dequantised products of the gate and up weights (epilogue_f64 of their
    exact accumulators), combined in fp64 and rounded once.  Returns (h fp16 [M, I], g, u).
    """
    g = epilogue_f64(gemm_exact(qa, qw_gate), a_alpha, a_beta, wa_gate, rs_gate, bias_gate)
    u = epilogue_f64(gemm_exact(qa, qw_up), a_alpha, a_beta, wa_up, rs_up, bias_up)
    return (silu(g) * u).astype(np.float16), g, u


def rotated_linear(x, w, had_dense=None, pow2_n: int = 1, bias=None):
    """The whole layer: had_quant_act -> pack_w4 -> GEMM -> epilogue.  Returns a dict."""
    xp, xa, xb, xr, qa = had_quant_act(x, had_dense, pow2_n)
    wp, wa, rs, qw = pack_w4(w, had_dense, pow2_n)
    y, acc = w4a4_linear(qa, xa[:, 0], xb[:, 0], qw, wa, rs, bias)
    return dict(x_packed=xp, x_alpha=xa[:, 0], x_beta=xb[:, 0], x_rot=xr, qa=qa,
                w_packed=wp, w_alpha=wa, w_rowsum=rs, qw=qw, acc=acc, y=y)


def reference_fp(x, w, bias=None) -> np.ndarray:
    """Unquantized fp64 x W^T (+ bias): for signal-to-noise reporting, not parity."""
    y = np.asarray(x, dtype=np.float64) @ np.asarray(w, dtype=np.float64).T
    if bias is not None:
        y = y + np.asarray(bias, dtype=np.float64)
    return y
