"""Round-to-nearest min-max quantizer of eq. 1 (Sec. 2) and 4-bit nibble packing.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Eq. 1:  X_Q = alpha * round((X_R - beta) / alpha) + beta, with
  symmetric:  alpha = max|X_R| / (2^(N-1) - 1),  beta = 0   -> codes in [-(2^(N-1)-1), 2^(N-1)-1]
  asymmetric: alpha = (max X_R - min X_R) / (2^N - 1), beta = min X_R -> codes in [0, 2^N - 1]
The paper quantizes activations and the KV cache asymmetrically with no range clipping
(App. A, "Quantization choice", Table 12) and weights symmetrically.

Readings of points the paper leaves open:
  * "round" is round-to-nearest with ties to even (np.rint).
  * beta is the real minimum, kept in fp32 (not an integer zero-point).
  * A group whose alpha = range / L would be zero or subnormal in fp32 (range below
    L * 2^-126, e.g. a constant group or an all-zero symmetric row) is treated as
    constant: alpha = 1 and every code 0, so it dequantizes to beta (exactly for a
    constant group, within the range otherwise).  This keeps 1 / alpha finite.
  * The encoding is carried out as this exact fp32 op sequence, one IEEE rounding per
    step, so that an implementation doing the same steps reproduces the codes bit for
    bit from the same fp32 inputs:
      asym: mn, mx = min, max;  r = mx - mn;  alpha = r / L (1 if that is below 2^-126);
            inv = 1 / alpha;  q = clamp(rint((v - mn) * inv), 0, L),  L = 2^N - 1
      sym:  a = max|v|;  alpha = a / L (1 if that is below 2^-126);  inv = 1 / alpha;
            q = clamp(rint(v * inv), -L, L),  L = 2^(N-1) - 1
    (dividing by alpha through its fp32 reciprocal is part of this reading).
"""

import numpy as np

F32 = np.float32
TINY = F32(np.finfo(np.float32).tiny)  # 2^-126, the smallest normal fp32


def _groups(v: np.ndarray, group: int) -> np.ndarray:
    K = v.shape[-1]
    if group <= 0 or K % group != 0:
        raise ValueError(f"group {group} does not divide row length {K}")
    return v.reshape(*v.shape[:-1], K // group, group)


F16_MAX = F32(65504.0)  # largest finite fp16


def to_fp16_sat(x: np.ndarray) -> np.ndarray:
    """fp32 -> fp16, round to nearest even, saturating at +-65504 instead of overflowing."""
    return np.clip(np.asarray(x, dtype=F32), -F16_MAX, F16_MAX).astype(np.float16)


def asym_codes(v: np.ndarray, alpha: np.ndarray, beta: np.ndarray, bits: int = 4,
               group: int | None = None) -> np.ndarray:
    """Codes of eq. 1 for given per-group parameters (fp32 or fp16 arrays [..., K/group]):
    inv = fl32(1 / alpha), q = clamp(rint(fl32(fl32(v - beta) * inv)), 0, 2^N - 1)."""
    v32 = np.asarray(v, dtype=F32)
    group = v32.shape[-1] if group is None else group
    g = _groups(v32, group)
    a32 = np.asarray(alpha).astype(F32).reshape(g.shape[:-1])
    b32 = np.asarray(beta).astype(F32).reshape(g.shape[:-1])
    inv = (F32(1) / a32).astype(F32)
    t = ((g - b32[..., None]).astype(F32) * inv[..., None]).astype(F32)
    return np.clip(np.rint(t), 0, 2 ** bits - 1).astype(np.int64).reshape(v32.shape)


def quant_asym(v: np.ndarray, bits: int = 4, group: int | None = None, clip: float = 1.0,
               param_fp16: bool = False):
    """Asymmetric min-max quantization of eq. 1 over contiguous groups of the last axis.

    v: fp32-representable values [..., K].  Returns (codes int64 [..., K] in [0, 2^N-1],
    alpha fp32 [..., K/group], beta fp32 [..., K/group]).
    clip < 1 quantizes the range [clip * min, clip * max] (each end rounded to fp32; the
    range clipping ablated in App. A "Quantization choice"); codes outside it clamp.
    param_fp16 stores alpha and beta as fp16 (returned as float16 arrays).  Reading: they
    are computed in fp32 as above, then rounded to fp16 (to_fp16_sat); a group whose fp32
    alpha is below 2^-126 or whose fp16 alpha is 0 is constant (alpha 1, codes 0); and the
    codes are taken from the stored pair, inv = fl32(1 / alpha16),
    q = clamp(rint(fl32(fl32(v - beta16) * inv)), 0, L), so that they dequantize to the
    nearest level of what is stored.
    """
    v32 = np.asarray(v, dtype=F32)
    group = v32.shape[-1] if group is None else group
    g = _groups(v32, group)
    levels = F32(2 ** bits - 1)
    mn = g.min(axis=-1)
    mx = g.max(axis=-1)
    if clip != 1.0:
        mn = (mn * F32(clip)).astype(F32)
        mx = (mx * F32(clip)).astype(F32)
    r = (mx - mn).astype(F32)
    alpha = (r / levels).astype(F32)
    if param_fp16:
        a16 = to_fp16_sat(alpha)
        a16 = np.where((alpha < TINY) | (a16 == 0), np.float16(1), a16).astype(np.float16)
        b16 = to_fp16_sat(mn)
        return asym_codes(v32, a16, b16, bits, group), a16, b16
    alpha = np.where(alpha < TINY, F32(1), alpha).astype(F32)
    return asym_codes(v32, alpha, mn, bits, group), alpha, mn.astype(F32)


def quant_sym(v: np.ndarray, bits: int = 4, group: int | None = None):
    """Symmetric quantization of eq. 1 (beta = 0) over contiguous groups of the last axis.

    Returns (codes int64 in [-(2^(N-1)-1), 2^(N-1)-1], alpha fp32 [..., K/group]).
    """
    v32 = np.asarray(v, dtype=F32)
    group = v32.shape[-1] if group is None else group
    g = _groups(v32, group)
    levels = F32(2 ** (bits - 1) - 1)
    amax = np.abs(g).max(axis=-1)
    alpha = (amax / levels).astype(F32)
    alpha = np.where(alpha < TINY, F32(1), alpha).astype(F32)
    inv = (F32(1) / alpha).astype(F32)
    t = (g * inv[..., None]).astype(F32)
    q = np.clip(np.rint(t), -levels, levels).astype(np.int64)
    return q.reshape(v32.shape), alpha


def dequant(q: np.ndarray, alpha: np.ndarray, beta: np.ndarray | None = None,
            group: int | None = None) -> np.ndarray:
    """X_Q = alpha * q + beta (eq. 1), in fp64, broadcasting per group."""
    q64 = np.asarray(q, dtype=np.float64)
    group = q64.shape[-1] if group is None else group
    g = _groups(q64, group)
    out = g * np.asarray(alpha, dtype=np.float64)[..., None]
    if beta is not None:
        out = out + np.asarray(beta, dtype=np.float64)[..., None]
    return out.reshape(q64.shape)


def pack_nibbles(q: np.ndarray) -> np.ndarray:
    """Two 4-bit codes per byte along the last axis: even index in the low nibble.

    Negative codes are stored as two's-complement nibbles.
    """
    qi = np.asarray(q, dtype=np.int64)
    if qi.shape[-1] % 2:
        raise ValueError("row length must be even to pack nibbles")
    lo = qi[..., 0::2] & 0xF
    hi = qi[..., 1::2] & 0xF
    return (lo | (hi << 4)).astype(np.uint8)


def store_codes(q: np.ndarray, bits: int) -> np.ndarray:
    """Storage of unsigned asymmetric codes: two per byte for 4 bits (pack_nibbles), one
    per byte for 8 bits (the W4A8 and KV8 settings of Sec. 4.2 "Main results" and of the
    speed measurement, Sec. 4.5)."""
    if bits == 4:
        return pack_nibbles(q)
    if bits == 8:
        return np.asarray(q, dtype=np.int64).astype(np.uint8)
    raise ValueError(f"no storage for {bits}-bit codes")


def unpack_nibbles(p: np.ndarray, signed: bool) -> np.ndarray:
    """Inverse of pack_nibbles: uint8 [..., K/2] -> int64 codes [..., K]."""
    b = np.asarray(p, dtype=np.int64)
    lo = b & 0xF
    hi = (b >> 4) & 0xF
    if signed:
        lo = np.where(lo >= 8, lo - 16, lo)
        hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty((*b.shape[:-1], 2 * b.shape[-1]), dtype=np.int64)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out
