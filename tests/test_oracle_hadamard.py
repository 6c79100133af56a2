"""Pins of the oracle's Hadamard constructions (test infrastructure checks, CPU only).

Fixed by the paper: a Hadamard matrix has +-1 entries and H/sqrt(n) is orthonormal
(Sec. 2.2 footnote; Sec. 3.2).  Sylvester is pinned to scipy's library routine, the
butterfly (fast Walsh-Hadamard transform, which the GPU kernels use) to the dense
Sylvester matrix by brute force.
"""

import numpy as np
import pytest
import scipy.linalg

from oracle import hadamard


@pytest.mark.parametrize("b", [1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024])
def test_sylvester_matches_scipy(b):
    assert np.array_equal(hadamard.sylvester(b).astype(np.int64), scipy.linalg.hadamard(b))


@pytest.mark.parametrize("n", [1, 28, 172])
def test_dense_factor_is_hadamard(n):
    h = hadamard.dense_factor(n).astype(np.int64)
    assert h.shape == (n, n)
    assert np.all(np.abs(h) == 1)
    assert np.array_equal(h @ h.T, n * np.eye(n, dtype=np.int64))
    assert np.array_equal(h.T @ h, n * np.eye(n, dtype=np.int64))


def test_paley_28_is_symmetric():
    h = hadamard.paley2(13).astype(np.int64)
    assert np.array_equal(h, h.T)


def test_paley_rejects_bad_q():
    with pytest.raises(ValueError):
        hadamard.paley2(7)  # 7 = 3 mod 4
    with pytest.raises(ValueError):
        hadamard.paley2(9)  # not prime


def test_williamson_blocks_are_symmetric_circulants():
    h = hadamard.williamson(43).astype(np.int64)
    m = 43
    A, B, C, D = h[:m, :m], h[:m, m:2 * m], h[:m, 2 * m:3 * m], h[:m, 3 * m:]
    for X in (A, B, C, D):
        assert np.array_equal(X, X.T)
        for i in range(1, m):
            assert np.array_equal(X[i], np.roll(X[0], i))
    # second block row of the Williamson array: [-B, A, -D, C]
    assert np.array_equal(h[m:2 * m], np.hstack([-B, A, -D, C]))


def test_williamson_is_deterministic():
    assert np.array_equal(hadamard.williamson(43), hadamard.williamson(43))


def test_check_rejects_perturbed_matrix():
    h = hadamard.dense_factor(28).copy()
    h[3, 5] = -h[3, 5]
    with pytest.raises(ValueError):
        hadamard.check(h)


def _fwht(v):
    """Plain in-place butterfly, natural (Hadamard) order."""
    v = np.array(v, dtype=np.float64)
    n = v.shape[-1]
    h = 1
    while h < n:
        for i in range(0, n, 2 * h):
            a = v[..., i:i + h].copy()
            b = v[..., i + h:i + 2 * h].copy()
            v[..., i:i + h] = a + b
            v[..., i + h:i + 2 * h] = a - b
        h *= 2
    return v


@pytest.mark.parametrize("n", [1, 2, 4, 8, 16, 32, 64])
def test_butterfly_equals_dense_sylvester_bruteforce(n):
    # the FWHT applied to each unit vector reproduces the rows of S_n
    eye = np.eye(n)
    assert np.array_equal(_fwht(eye), hadamard.sylvester(n).astype(np.float64))
    rng = np.random.default_rng(n)
    x = rng.standard_normal((5, n))
    np.testing.assert_allclose(_fwht(x), x @ hadamard.sylvester(n).astype(np.float64), rtol=0, atol=1e-12)
