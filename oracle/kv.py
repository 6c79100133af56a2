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

from .quant import pack_nibbles, quant_asym
from .rotate import rotate_rows


def qk_had_kvquant(q: np.ndarray, k: np.ndarray, v: np.ndarray, bits: int = 4, group: int = 128):
    """q, k, v: fp16 [B, S, H, D].  Returns a dict with
    q_rot fp16 [B,S,H,D]; k_rot fp32 (quantizer input);
    k_q, v_q uint8 [B,S,H,D/2]; k_alpha, k_beta, v_alpha, v_beta fp32 [B,S,H,D/group];
    k_codes, v_codes int64 [B,S,H,D].
    """
    D = q.shape[-1]
    q_rot = rotate_rows(q, None, D).astype(np.float16)
    k_rot = rotate_rows(k, None, D).astype(np.float32)
    kc, ka, kb = quant_asym(k_rot, bits=bits, group=group)
    vc, va, vb = quant_asym(np.asarray(v, dtype=np.float32), bits=bits, group=group)
    return dict(q_rot=q_rot, k_rot=k_rot, k_q=pack_nibbles(kc), k_alpha=ka, k_beta=kb,
                v_q=pack_nibbles(vc), v_alpha=va, v_beta=vb, k_codes=kc, v_codes=vc)
