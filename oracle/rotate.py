"""Online Hadamard rotation of activation rows (R4 on the down-projection input, R3 on
post-RoPE Q and K), Sec. 3.1 "Additional unabsorbed rotations".

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper fixes the rotation as a Hadamard matrix applied online and scaled to be
orthonormal (Sec. 2.2 footnote, Sec. 3.2).  For a width n = a * b that is not a power
of two, the rotation used here is the Kronecker product R = (H_a (x) S_b) / sqrt(n),
with H_a a dense Hadamard factor of order a and S_b the Sylvester matrix of order
b = 2^k.  Reading of the paper (it is silent on the order of the Kronecker factors): the
dense factor acts on the outer, strided index and the Sylvester factor on the inner,
contiguous one, i.e. element i of a block is (i_a, i_b) with i = i_a * b + i_b.  Rows
are row vectors, as the paper writes X R_1 in Sec. 3.1:  y = x R.  When n < K each
contiguous n-block of a row is rotated on its own (block-diagonal I (x) R).

The product is computed in fp64 with the dense factors:
    X2 = x.reshape(a, b);  Y2 = H_a^T X2 S_b;  y = Y2.reshape(n) / sqrt(n)
which equals x (H_a (x) S_b) / sqrt(n) element for element.
"""

import numpy as np

from .hadamard import sylvester


def rotation_matrix(had_dense: np.ndarray | None, pow2_n: int) -> np.ndarray:
    """The dense fp64 orthonormal rotation (H_a (x) S_b) / sqrt(n)."""
    ha = np.ones((1, 1)) if had_dense is None else had_dense.astype(np.float64)
    sb = sylvester(pow2_n).astype(np.float64)
    r = np.kron(ha, sb)
    return r / np.sqrt(r.shape[0])


def rotate_rows(x: np.ndarray, had_dense: np.ndarray | None, pow2_n: int) -> np.ndarray:
    """y = x (H_a (x) S_b) / sqrt(n) for each contiguous n-block of each row, in fp64.

    x: [..., K] any real dtype (converted exactly to fp64); n = a * pow2_n must
    divide K.  Returns fp64 [..., K].
    """
    x64 = np.asarray(x, dtype=np.float64)
    a = 1 if had_dense is None else had_dense.shape[0]
    b = int(pow2_n)
    n = a * b
    K = x64.shape[-1]
    if K % n != 0:
        raise ValueError(f"rotation width {n} does not divide row length {K}")
    ha = np.ones((1, 1)) if had_dense is None else had_dense.astype(np.float64)
    sb = sylvester(b).astype(np.float64)
    lead = x64.shape[:-1]
    x2 = x64.reshape(-1, K // n, a, b)
    # Y2 = H_a^T X2 S_b for every block
    y2 = np.matmul(np.matmul(ha.T, x2), sb)
    return (y2 / np.sqrt(n)).reshape(*lead, K)
