"""R3 on post-RoPE queries and keys, then 4-bit asymmetric K/V cache quantization.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 3.1 ("Additional unabsorbed rotations") inserts the online Hadamard R3 in the
attention block when the KV cache is quantized to low bits.  It is applied head by
head to Q and K after RoPE: (Q R)(K R)^T = Q K^T because R is orthonormal, so the
attention scores are unchanged in full precision.  V is not rotated online (its
rotation R2 is merged into W_v offline, Sec. 3.1).  The cache is quantized
asymmetrically without clipping (App. A "Quantization choice", Table 12).  The group
is the head dimension of one (batch, token, head), D = 128 elements (a reading: the
paper does not state the KV group size).
"""

import numpy as np

from .quant import dequant, pack_nibbles, quant_asym, store_codes, unpack_nibbles
from .rotate import rotate_rows


def qk_had_kvquant(q: np.ndarray, k: np.ndarray, v: np.ndarray, bits: int = 4, group: int = 128,
                   k_clip: float = 1.0, v_clip: float = 1.0, param_fp16: bool = False):
    """q, k, v: fp16 [B, S, H, D].  Returns a dict with
    q_rot fp16 [B,S,H,D]; k_rot fp32 (quantizer input);
    k_q, v_q uint8 [B,S,H,D/2] (bits 4) or [B,S,H,D] (bits 8);
    k_alpha, k_beta, v_alpha, v_beta fp32 (fp16 with param_fp16) [B,S,H,D/group];
    k_codes, v_codes int64 [B,S,H,D].
    k_clip, v_clip < 1 clip the groups' ranges (quant_asym; App. A uses 0.95 for the cache).
    param_fp16: the group parameters stored in fp16 (quant_asym), halving their share of
    the cache.
    """
    D = q.shape[-1]
    q_rot = rotate_rows(q, None, D).astype(np.float16)
    k_rot = rotate_rows(k, None, D).astype(np.float32)
    kc, ka, kb = quant_asym(k_rot, bits=bits, group=group, clip=k_clip, param_fp16=param_fp16)
    vc, va, vb = quant_asym(np.asarray(v, dtype=np.float32), bits=bits, group=group, clip=v_clip,
                            param_fp16=param_fp16)
    return dict(q_rot=q_rot, k_rot=k_rot, k_q=store_codes(kc, bits), k_alpha=ka, k_beta=kb,
                v_q=store_codes(vc, bits), v_alpha=va, v_beta=vb, k_codes=kc, v_codes=vc)


def attn_decode(q_rot, k_q, k_alpha, k_beta, v_q, v_alpha, v_beta, scale=None):
    """Attention of one new query per (batch, head) over the 4-bit cache written by
    qk_had_kvquant, the step that consumes it.

    Keys and values are dequantised by eq. 1, K_t = alpha_t c_t + beta_t (in the R3-rotated
    basis for K); the query is rotated the same way, so q_rot . K_t is the score of the
    unrotated pair up to the cache's quantization error (Sec. 3.1).
      q_rot   fp16 [B, H, D]
      k_q, v_q  uint8 [B, S, H, D/2]; alphas, betas fp32 or fp16 [B, S, H] (or [B, S, H, 1])
      scale   score scale, 1/sqrt(D) by default
    Returns fp16 [B, H, D] = fp16( softmax_t(scale q_rot . K_t) V ), fp64 inside.
    """
    D = q_rot.shape[-1]
    scale = 1.0 / np.sqrt(D) if scale is None else scale
    B, S, H = k_q.shape[:3]
    kc = unpack_nibbles(k_q, signed=False)
    vc = unpack_nibbles(v_q, signed=False)
    K = dequant(kc, np.reshape(k_alpha, (B, S, H, 1)), np.reshape(k_beta, (B, S, H, 1)), group=D)
    V = dequant(vc, np.reshape(v_alpha, (B, S, H, 1)), np.reshape(v_beta, (B, S, H, 1)), group=D)
    q = np.asarray(q_rot, dtype=np.float64)
    s = np.einsum("bhd,bshd->bhs", q, K) * scale
    p = np.exp(s - s.max(axis=-1, keepdims=True))
    p /= p.sum(axis=-1, keepdims=True)
    return np.einsum("bhs,bshd->bhd", p, V).astype(np.float16)
