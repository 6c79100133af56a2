"""Pins of the oracle's R3 + 4-bit KV-cache quantization (CPU only).

Fixed by the paper: R3 leaves the attention scores unchanged in full precision (Sec.
3.1); the cache is quantized asymmetrically (App. A Table 12) so each group's minimum
maps to 0 and maximum to 15 and every reconstruction is within alpha/2 of its input.
"""

import numpy as np

from oracle import kv, quant, rotate
from paper_2405_16406_amd import workloads


def _small():
    return workloads.kv_inputs(B=2, S=16, H=4, D=128)


def test_shapes_and_layout():
    q, k, v = _small()
    out = kv.qk_had_kvquant(q, k, v)
    assert out["q_rot"].shape == q.shape and out["q_rot"].dtype == np.float16
    assert out["k_q"].shape == (2, 16, 4, 64) and out["k_q"].dtype == np.uint8
    assert out["k_alpha"].shape == (2, 16, 4, 1)


def test_scores_preserved_by_r3_before_quantization():
    q, k, _ = _small()
    qr = rotate.rotate_rows(q, None, 128)
    kr = rotate.rotate_rows(k, None, 128)
    s0 = np.einsum("bshd,bthd->bhst", q.astype(np.float64), k.astype(np.float64))
    s1 = np.einsum("bshd,bthd->bhst", qr, kr)
    assert np.max(np.abs(s1 - s0)) <= 1e-10 * np.max(np.abs(s0))


def test_v_is_not_rotated_and_codes_exact():
    q, k, v = _small()
    out = kv.qk_had_kvquant(q, k, v)
    c, a, b = quant.quant_asym(v.astype(np.float32), group=128)
    np.testing.assert_array_equal(out["v_codes"], c)
    np.testing.assert_array_equal(out["v_alpha"], a)
    np.testing.assert_array_equal(out["v_beta"], b)


def test_k_codes_bound_and_extremes():
    q, k, v = _small()
    out = kv.qk_had_kvquant(q, k, v)
    kc, ka, kb, kr = out["k_codes"], out["k_alpha"], out["k_beta"], out["k_rot"]
    assert kc.min() >= 0 and kc.max() <= 15
    err = np.abs(quant.dequant(kc, ka, kb, group=128) - kr.astype(np.float64))
    assert np.all(err <= np.repeat(ka, 128, axis=-1) * 0.5 * (1 + 1e-6))
    flat = kr.reshape(-1, 128)
    codes = kc.reshape(-1, 128)
    assert np.all(codes[np.arange(flat.shape[0]), flat.argmin(1)] == 0)
    assert np.all(codes[np.arange(flat.shape[0]), flat.argmax(1)] == 15)


def test_r3_lowers_k_quant_error_with_outlier_dims():
    q, k, v = _small()
    out = kv.qk_had_kvquant(q, k, v)
    rot_err = np.mean((quant.dequant(out["k_codes"], out["k_alpha"], out["k_beta"], 128)
                       - out["k_rot"]) ** 2)
    c, a, b = quant.quant_asym(k.astype(np.float32), group=128)
    plain_err = np.mean((quant.dequant(c, a, b, 128) - k.astype(np.float64)) ** 2)
    assert rot_err < 0.5 * plain_err
