"""Pins of the oracle's rotated W4A4 linear layer (CPU only).

* exact integer GEMM == brute-force triple loop on tiny shapes;
* epilogue == dequant(qa) dequant(qw)^T, the algebraic expansion of eq. 1 on both
  operands, to 1e-12 in fp64 (catches a dropped zero-point term or a wrong sign);
* identity rotation == plain per-token quantization;
* rotating outlier activations raises the W4A4 signal-to-noise ratio (Sec. 2.1 Fig. 3,
  App. B.2 Table 19 direction).
"""

import numpy as np
import pytest

from oracle import hadamard, linear, quant, rotate
from paper_2405_16406_amd import workloads


def test_gemm_exact_bruteforce():
    rng = np.random.default_rng(0)
    qa = rng.integers(0, 16, size=(5, 24))
    qw = rng.integers(-7, 8, size=(6, 24))
    acc = linear.gemm_exact(qa, qw)
    for m in range(5):
        for n in range(6):
            s = 0
            for k in range(24):
                s += int(qa[m, k]) * int(qw[n, k])
            assert acc[m, n] == s


def test_gemm_exact_extreme_values():
    K = 28672
    qa = np.full((2, K), 15)
    qw = np.full((3, K), -7)
    acc = linear.gemm_exact(qa, qw)
    assert np.all(acc == -105 * K)


def test_epilogue_is_expanded_dequant_product():
    rng = np.random.default_rng(1)
    M, N, K = 7, 9, 64
    qa = rng.integers(0, 16, size=(M, K))
    qw = rng.integers(-7, 8, size=(N, K))
    aa = rng.uniform(0.1, 2.0, M).astype(np.float32)
    ab = rng.uniform(-5, 0, M).astype(np.float32)
    wa = rng.uniform(1e-3, 1e-2, N).astype(np.float32)
    rs = qw.sum(1).astype(np.int32)
    acc = linear.gemm_exact(qa, qw)
    y64 = linear.epilogue_f64(acc, aa, ab, wa, rs)
    ref = quant.dequant(qa, aa[:, None], ab[:, None]) @ quant.dequant(qw, wa[:, None]).T
    assert np.max(np.abs(y64 - ref)) <= 1e-12 * np.max(np.abs(ref))
    bias = rng.standard_normal(N).astype(np.float16)
    y = linear.epilogue(acc, aa, ab, wa, rs, bias)
    assert y.dtype == np.float16
    np.testing.assert_array_equal(y, (ref + bias.astype(np.float64)).astype(np.float16))


def test_identity_rotation_is_plain_per_token_quant():
    x, _ = workloads.tiny_inputs()
    p, a, b, y32, q = linear.had_quant_act(x, None, 1)
    q2, a2, b2 = quant.quant_asym(x.astype(np.float32))
    np.testing.assert_array_equal(q, q2)
    np.testing.assert_array_equal(a, a2)
    np.testing.assert_array_equal(b, b2)
    np.testing.assert_array_equal(p, quant.pack_nibbles(q2))


def test_pack_w4_rowsum_and_range():
    _, w = workloads.tiny_inputs()
    p, a, rs, q = linear.pack_w4(w, None, 256)
    assert q.min() >= -7 and q.max() <= 7
    np.testing.assert_array_equal(rs, q.sum(1))
    np.testing.assert_array_equal(quant.unpack_nibbles(p, signed=True), q)
    assert a.shape == (256,)


def _snr_db(ref, y):
    return 10 * np.log10(np.sum(ref ** 2) / np.sum((ref - y.astype(np.float64)) ** 2))


def test_rotation_improves_w4a4_snr():
    x, w = workloads.tiny_inputs()
    ref = linear.reference_fp(x, w)
    plain = linear.rotated_linear(x, w, None, 1)
    rot = linear.rotated_linear(x, w, None, 256)
    assert _snr_db(ref, rot["y"]) > _snr_db(ref, plain["y"]) + 3.0


def test_rotated_layer_kronecker_invariance_small():
    # the rotated layer approximates x W^T; with 8-bit-like fine steps it would be exact
    rng = np.random.default_rng(5)
    ha = hadamard.dense_factor(28)
    K = 28 * 8
    x = rng.standard_normal((6, K)).astype(np.float16)
    w = (0.02 * rng.standard_normal((10, K))).astype(np.float16)
    out = linear.rotated_linear(x, w, ha, 8)
    ref = linear.reference_fp(x, w)
    assert _snr_db(ref, out["y"]) > 10.0
    np.testing.assert_array_equal(out["acc"], linear.gemm_exact(out["qa"], out["qw"]))
    # the weight really was rotated with the same rotation as the activations
    wr = rotate.rotate_rows(w, ha, 8).astype(np.float32)
    q, a = quant.quant_sym(wr)
    np.testing.assert_array_equal(out["qw"], q)


@pytest.mark.parametrize("bits", [4, 8])
def test_had_quant_act_code_range(bits):
    x, _ = workloads.tiny_inputs()
    _, a, b, y32, q = linear.had_quant_act(x, None, 256, bits=bits)
    assert q.min() >= 0 and q.max() <= 2 ** bits - 1
    err = np.abs(quant.dequant(q, a, b) - y32.astype(np.float64))
    assert np.all(err <= a.astype(np.float64) * 0.5 * (1 + 1e-5))


def test_silu_closed_forms():
    # SiLU(v) = v sigma(v): sigma(0) = 1/2, sigma(ln 3) = 3/4, sigma(-ln 3) = 1/4, and
    # SiLU(v) - SiLU(-v) = v (sigma(v) + sigma(-v) = 1); large v tends to v, large -v to 0
    ln3 = np.log(3.0)
    v = linear.silu(np.array([0.0, ln3, -ln3, 2.0, -2.0, 40.0, -40.0, -800.0]))
    assert v[0] == 0.0
    assert abs(v[1] - 0.75 * ln3) < 1e-15 and abs(v[2] + 0.25 * ln3) < 1e-15
    assert abs((v[3] - v[4]) - 2.0) < 1e-15
    assert abs(v[5] - 40.0) < 1e-15 and abs(v[6]) < 1e-15
    assert v[7] == 0.0 and np.isfinite(v[7])


def test_swiglu_linear_bruteforce():
    # h[m, c] = fp16(SiLU(g) u) with g, u the dequantised gate/up products, element by element
    import math
    rng = np.random.default_rng(5)
    M, I, K = 3, 5, 16
    qa = rng.integers(0, 16, size=(M, K))
    aa, ab = rng.uniform(0.01, 0.1, M), rng.uniform(-1, 0, M)
    qg, qu = rng.integers(-7, 8, size=(I, K)), rng.integers(-7, 8, size=(I, K))
    ga, ua = rng.uniform(0.001, 0.01, I), rng.uniform(0.001, 0.01, I)
    bg, bu = rng.uniform(-0.1, 0.1, I), rng.uniform(-0.1, 0.1, I)
    h, g, u = linear.swiglu_linear(qa, aa, ab, qg, ga, qg.sum(1), qu, ua, qu.sum(1), bg, bu)
    for m in range(M):
        for c in range(I):
            gv = sum((aa[m] * qa[m, k] + ab[m]) * ga[c] * qg[c, k] for k in range(K)) + bg[c]
            uv = sum((aa[m] * qa[m, k] + ab[m]) * ua[c] * qu[c, k] for k in range(K)) + bu[c]
            assert abs(g[m, c] - gv) < 1e-12 and abs(u[m, c] - uv) < 1e-12
            ref = gv / (1.0 + math.exp(-gv)) * uv
            assert h[m, c] == np.float16(ref)


def test_w4a8_gemm_and_epilogue_bruteforce():
    # 8-bit activation codes against 4-bit weights: the same exact GEMM and epilogue
    rng = np.random.default_rng(6)
    qa = rng.integers(0, 256, size=(3, 40))
    qw = rng.integers(-7, 8, size=(4, 40))
    aa, ab = rng.uniform(0.01, 0.1, 3), rng.uniform(-3, 0, 3)
    wa = rng.uniform(0.001, 0.01, 4)
    y, acc = linear.w4a4_linear(qa, aa, ab, qw, wa, qw.sum(1))
    for m in range(3):
        for n in range(4):
            s = sum(int(qa[m, k]) * int(qw[n, k]) for k in range(40))
            assert acc[m, n] == s
            ref = sum((aa[m] * qa[m, k] + ab[m]) * (wa[n] * qw[n, k]) for k in range(40))
            assert y[m, n] == np.float16(ref)


def test_had_quant_act_8bit_storage():
    x = workloads.outlier_acts(workloads.rng_for(12), 4, 256, 4, 50.0)
    p8, a8, b8, y8, q8 = linear.had_quant_act(x, None, 256, bits=8)
    assert p8.shape == (4, 256) and p8.dtype == np.uint8 and np.array_equal(p8.astype(np.int64), q8)
    assert q8.min() == 0 and q8.max() == 255


def test_random_sign_hadamard_rotation():
    # R = S (H_28 (x) S_4) / sqrt(112) with a random +-1 diagonal S is orthonormal; all-plus
    # signs give the plain rotation; folding the same R into the weights keeps x W^T
    rng = np.random.default_rng(13)
    had = hadamard.dense_factor(28)
    s = rng.choice([-1, 1], 112).astype(np.int8)
    R = rotate.rotate_rows(np.diag(s.astype(np.float64)), had, 4)      # rows of S H / sqrt(n)
    np.testing.assert_allclose(R @ R.T, np.eye(112), atol=1e-12)
    x = rng.standard_normal((3, 224)).astype(np.float16)
    plus = np.ones(112, np.int8)
    np.testing.assert_array_equal(linear.had_quant_act(x, had, 4, signs=plus)[3], linear.had_quant_act(x, had, 4)[3])
    y = linear.had_quant_act(x, had, 4, signs=s)[3].astype(np.float64)
    x64 = x.astype(np.float64)
    np.testing.assert_allclose(y[:, :112], x64[:, :112] @ R, rtol=0, atol=1e-5 * np.abs(y).max())
    w = rng.standard_normal((5, 224)).astype(np.float16)
    wr = linear._signed(w, s, 112)
    wr = rotate.rotate_rows(wr, had, 4)
    yr = rotate.rotate_rows(linear._signed(x, s, 112), had, 4)
    np.testing.assert_allclose(yr @ wr.T, x64 @ w.astype(np.float64).T, rtol=0, atol=1e-10 * 224)
