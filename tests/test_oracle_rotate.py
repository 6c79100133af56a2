"""Pins of the oracle's row rotation (CPU only).

Fixed by the paper: the rotation is orthonormal, so a full-precision network is
unchanged, (x R)(W R)^T = x W^T (Sec. 3.1; App. B.1 shows the gradient through R is
zero without quantization) and (Q R)(K R)^T = Q K^T head by head; rotating outlier
activations drives their kurtosis to about 3 (Sec. 2.1, Fig. 3).  The index
convention of the reshape formulation is pinned to an explicit np.kron.
"""

import numpy as np
import pytest

from oracle import hadamard, rotate


@pytest.mark.parametrize("a,b,blocks", [(1, 1, 3), (1, 8, 2), (1, 256, 1), (28, 4, 2), (28, 2, 1),
                                        (172, 2, 1), (172, 1, 2)])
def test_reshape_form_equals_explicit_kronecker(a, b, blocks):
    ha = None if a == 1 else hadamard.dense_factor(a)
    n = a * b
    rng = np.random.default_rng(a * 1000 + b)
    x = rng.standard_normal((4, n * blocks))
    y = rotate.rotate_rows(x, ha, b)
    ha64 = np.ones((1, 1)) if ha is None else ha.astype(np.float64)
    R = np.kron(ha64, hadamard.sylvester(b).astype(np.float64)) / np.sqrt(n)
    expect = np.concatenate([x[:, i * n:(i + 1) * n] @ R for i in range(blocks)], axis=1)
    np.testing.assert_allclose(y, expect, rtol=0, atol=1e-12)


def test_reshape_index_convention_unit_vector():
    # e_{i_a*b + i_b} maps to row (i_a, i_b) of H_a (x) S_b: y[j_a*b + j_b] = H[i_a,j_a] S[i_b,j_b]/sqrt(n)
    ha = hadamard.dense_factor(28)
    b = 4
    n = 28 * b
    i_a, i_b = 5, 2
    x = np.zeros((1, n))
    x[0, i_a * b + i_b] = 1.0
    y = rotate.rotate_rows(x, ha, b)[0].reshape(28, b)
    S = hadamard.sylvester(b).astype(np.float64)
    expect = np.outer(ha[i_a].astype(np.float64), S[i_b]) / np.sqrt(n)
    np.testing.assert_allclose(y, expect, rtol=0, atol=1e-15)


@pytest.mark.parametrize("b", [2, 64, 256])
def test_constant_row_closed_form(b):
    # sum of the rows of a natural-order Sylvester matrix is b * e_0:  c*1 -> c*sqrt(b)*e_0
    x = np.full((1, b), 0.75)
    y = rotate.rotate_rows(x, None, b)[0]
    expect = np.zeros(b)
    expect[0] = 0.75 * np.sqrt(b)
    np.testing.assert_allclose(y, expect, rtol=0, atol=1e-13)


@pytest.mark.parametrize("a,b", [(1, 256), (28, 16), (172, 4)])
def test_rotation_is_orthonormal(a, b):
    ha = None if a == 1 else hadamard.dense_factor(a)
    R = rotate.rotation_matrix(ha, b)
    np.testing.assert_allclose(R @ R.T, np.eye(a * b), rtol=0, atol=1e-12)


@pytest.mark.parametrize("a,b", [(28, 8), (172, 2), (1, 128)])
def test_rotational_invariance_of_linear_layer(a, b):
    ha = None if a == 1 else hadamard.dense_factor(a)
    K = a * b * 2
    rng = np.random.default_rng(7)
    x = rng.standard_normal((8, K))
    x[:, rng.choice(K, 4, replace=False)] *= 50.0
    w = 0.02 * rng.standard_normal((16, K))
    y0 = x @ w.T
    y1 = rotate.rotate_rows(x, ha, b) @ rotate.rotate_rows(w, ha, b).T
    assert np.max(np.abs(y1 - y0)) <= 1e-10 * np.max(np.abs(y0))


def test_attention_scores_invariant_per_head():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((2, 5, 4, 128))
    k = rng.standard_normal((2, 5, 4, 128))
    qr = rotate.rotate_rows(q, None, 128)
    kr = rotate.rotate_rows(k, None, 128)
    s0 = np.einsum("bshd,bthd->bhst", q, k)
    s1 = np.einsum("bshd,bthd->bhst", qr, kr)
    np.testing.assert_allclose(s1, s0, rtol=0, atol=1e-10 * np.abs(s0).max())


def test_norm_preserved():
    ha = hadamard.dense_factor(172)
    rng = np.random.default_rng(11)
    x = rng.standard_normal((3, 172 * 64))
    y = rotate.rotate_rows(x, ha, 64)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-12)


def test_rejects_non_dividing_width():
    with pytest.raises(ValueError):
        rotate.rotate_rows(np.zeros((1, 100)), hadamard.dense_factor(28), 2)


def _kurtosis(v):
    v = v - v.mean()
    return float(np.mean(v ** 4) / np.mean(v ** 2) ** 2)


def test_rotation_drives_kurtosis_to_gaussian():
    # Sec. 2.1 / Fig. 3(a): outlier channels give kurtosis >> 3; after rotation ~ 3
    rng = np.random.default_rng(0)
    K = 28 * 64
    x = rng.standard_normal((64, K))
    x[:, rng.choice(K, int(0.01 * K), replace=False)] *= 50.0
    k0 = _kurtosis(x.ravel())
    k1 = _kurtosis(rotate.rotate_rows(x, hadamard.dense_factor(28), 64).ravel())
    assert k0 > 50
    assert abs(k1 - 3.0) < 0.3
