"""Pins of the oracle's quantizer and packing (CPU only).

Fixed by the paper (Sec. 2, eq. 1): asymmetric min-max maps the minimum to code 0 and
the maximum to 2^N - 1; symmetric maps +-max|x| to +-(2^(N-1) - 1); round-to-nearest
keeps every reconstruction within alpha/2; App. A Table 12 prefers asymmetric
quantization for activations and the KV cache.  Hand-worked cases in
tests/golden/quant_worked.json pin the tie rule and the scale/offset values.
"""

import json
import os

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st
from hypothesis.extra.numpy import arrays

from oracle import quant

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "quant_worked.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.mark.parametrize("case", _golden()["asym"])
def test_asym_golden(case):
    q, a, b = quant.quant_asym(np.array(case["v"], dtype=np.float32), bits=case["bits"])
    assert q.tolist() == case["codes"]
    assert a == np.float32(case["alpha"])
    assert b == np.float32(case["beta"])


@pytest.mark.parametrize("case", _golden()["sym"])
def test_sym_golden(case):
    q, a = quant.quant_sym(np.array(case["v"], dtype=np.float32), bits=case["bits"])
    assert q.tolist() == case["codes"]
    assert a == np.float32(case["alpha"])


def test_asym_closed_forms_and_bound():
    rng = np.random.default_rng(0)
    v = (rng.standard_normal((50, 256)) * 3 + 1).astype(np.float32)
    q, a, b = quant.quant_asym(v, bits=4)
    assert q.min() >= 0 and q.max() <= 15
    assert np.all(q[np.arange(50), v.argmin(1)] == 0)
    assert np.all(q[np.arange(50), v.argmax(1)] == 15)
    np.testing.assert_array_equal(b[:, 0], v.min(1))
    vhat = quant.dequant(q, a, b)
    err = np.abs(vhat - v.astype(np.float64))
    assert np.all(err <= a.astype(np.float64) * 0.5 * (1 + 1e-6))


def test_asym_groups_are_independent():
    rng = np.random.default_rng(1)
    v = rng.standard_normal((4, 512)).astype(np.float32)
    q, a, b = quant.quant_asym(v, bits=4, group=128)
    assert a.shape == (4, 4) and b.shape == (4, 4)
    for g in range(4):
        qg, ag, bg = quant.quant_asym(v[:, g * 128:(g + 1) * 128], bits=4)
        np.testing.assert_array_equal(q[:, g * 128:(g + 1) * 128], qg)
        np.testing.assert_array_equal(a[:, g], ag[:, 0])
        np.testing.assert_array_equal(b[:, g], bg[:, 0])


def test_sym_closed_forms_and_bound():
    rng = np.random.default_rng(2)
    w = (rng.standard_normal((40, 300)) * 0.02).astype(np.float32)
    q, a = quant.quant_sym(w, bits=4)
    assert q.min() >= -7 and q.max() <= 7
    i = np.abs(w).argmax(1)
    np.testing.assert_array_equal(q[np.arange(40), i], np.sign(w[np.arange(40), i]) * 7)
    err = np.abs(quant.dequant(q, a) - w.astype(np.float64))
    assert np.all(err <= a.astype(np.float64) * 0.5 * (1 + 1e-6))


def test_degenerate_groups():
    v = np.full((2, 8), -2.5, dtype=np.float32)
    q, a, b = quant.quant_asym(v)
    assert np.all(q == 0) and np.all(a == 1) and np.all(b == np.float32(-2.5))
    np.testing.assert_array_equal(quant.dequant(q, a, b), v)
    q, a = quant.quant_sym(np.zeros((2, 8), dtype=np.float32))
    assert np.all(q == 0) and np.all(a == 1)


def test_asym_beats_sym_on_rotated_activations():
    # App. A Table 12: asymmetric activation quantization is the better choice
    rng = np.random.default_rng(4)
    v = (rng.standard_normal((256, 512)) + 0.4).astype(np.float32)
    qa, aa, ba = quant.quant_asym(v)
    qs, as_ = quant.quant_sym(v)
    ea = np.mean((quant.dequant(qa, aa, ba) - v) ** 2)
    es = np.mean((quant.dequant(qs, as_) - v) ** 2)
    assert ea < es


def test_tiny_range_is_constant():
    # alpha = range / L below the smallest normal fp32 would make 1 / alpha overflow: the
    # group is quantized as constant (alpha 1, codes 0) and dequantizes to beta, within the range.
    tiny = np.finfo(np.float32).tiny
    for top in [np.float32(8.76e-43), np.float32(1e-37), np.float32(15 * tiny * 0.999)]:
        v = np.array([[top, 0, 0, 0]], dtype=np.float32)
        q, a, b = quant.quant_asym(v, bits=4)
        assert a[0, 0] == 1 and b[0, 0] == 0 and not q.any()
        assert np.abs(quant.dequant(q, a, b) - v).max() <= top
    for top in [np.float32(8.76e-43), np.float32(5e-38), np.float32(7 * tiny * 0.999)]:
        qs, as_ = quant.quant_sym(np.array([[top, -top / 2, 0, 0]], dtype=np.float32), bits=4)
        assert as_[0, 0] == 1 and not qs.any()
    # just above the threshold the quantizer works normally
    v = np.array([[np.float32(16 * tiny), 0, 0, 0]], dtype=np.float32)
    q, a, b = quant.quant_asym(v, bits=4)
    assert a[0, 0] >= tiny and q.tolist() == [[15, 0, 0, 0]]


def test_pack_layout_and_roundtrip():
    q = np.array([[1, 2, 15, 0, 7, 8]])
    p = quant.pack_nibbles(q)
    assert p.tolist() == [[0x21, 0x0F, 0x87]]
    np.testing.assert_array_equal(quant.unpack_nibbles(p, signed=False), q)
    s = np.array([[-7, 7, -1, 0, 3, -4]])
    ps = quant.pack_nibbles(s)
    assert ps.tolist() == [[0x79, 0x0F, 0xC3]]
    np.testing.assert_array_equal(quant.unpack_nibbles(ps, signed=True), s)


@settings(max_examples=200, deadline=None)
@given(arrays(np.float32, st.integers(2, 64).map(lambda n: (2 * n,)),
              elements=st.floats(-1e4, 1e4, width=32, allow_nan=False, allow_infinity=False)))
def test_asym_properties(v):
    q, a, b = quant.quant_asym(v[None, :], bits=4)
    assert q.min() >= 0 and q.max() <= 15
    assert b[0, 0] == v.min()
    r = np.float32(v.max() - v.min())
    if r / np.float32(15) >= np.finfo(np.float32).tiny:
        assert q[0, v.argmin()] == 0 and q[0, v.argmax()] == 15
        err = np.abs(quant.dequant(q, a, b)[0] - v.astype(np.float64))
        # alpha/2 plus the fp32 rounding of (v - min) * (1/alpha)
        assert np.all(err <= np.float64(a[0, 0]) * (0.5 + 4e-6) + 1e-6 * np.abs(v).max())
    p = quant.pack_nibbles(q)
    np.testing.assert_array_equal(quant.unpack_nibbles(p, signed=False), q)


@settings(max_examples=200, deadline=None)
@given(arrays(np.float32, st.integers(1, 64).map(lambda n: (2 * n,)),
              elements=st.floats(-100, 100, width=32, allow_nan=False, allow_infinity=False)))
def test_sym_properties(v):
    q, a = quant.quant_sym(v[None, :], bits=4)
    assert q.min() >= -7 and q.max() <= 7
    amax = np.abs(v).max()
    if amax / np.float32(7) >= np.finfo(np.float32).tiny:
        assert abs(q[0, np.abs(v).argmax()]) == 7
        err = np.abs(quant.dequant(q, a)[0] - v.astype(np.float64))
        assert np.all(err <= np.float64(a[0, 0]) * (0.5 + 4e-6))
    np.testing.assert_array_equal(quant.unpack_nibbles(quant.pack_nibbles(q), signed=True), q)


def test_asym_8bit_closed_forms_and_storage():
    # 8-bit asymmetric codes (the W4A8 / KV8 settings): min -> 0, max -> 255, every
    # reconstruction within alpha/2, a linear ramp hits every level once, one code per byte
    v = np.linspace(-3.0, 5.0, 256, dtype=np.float32)[None, :]
    q, a, b = quant.quant_asym(v, bits=8)
    np.testing.assert_array_equal(q[0], np.arange(256))
    assert a[0] == np.float32(np.float32(8.0) / np.float32(255.0)) and b[0] == np.float32(-3.0)
    rng = np.random.default_rng(8)
    x = (rng.standard_normal((5, 96)) * 4).astype(np.float32)
    q, a, b = quant.quant_asym(x, bits=8, group=32)
    assert q.min() >= 0 and q.max() <= 255
    err = np.abs(quant.dequant(q, a, b, group=32) - x.astype(np.float64))
    assert np.all(err <= np.repeat(a, 32, axis=-1) * 0.5 * (1 + 1e-6))
    s = quant.store_codes(q, 8)
    assert s.dtype == np.uint8 and s.shape == q.shape and np.array_equal(s.astype(np.int64), q)
    with pytest.raises(ValueError):
        quant.store_codes(q, 6)


def test_asym_clip_closed_form():
    # clip r: the range [r min, r max]; a ramp on [-4, 4] with r = 0.5 quantizes [-2, 2]:
    # alpha = 4/15, beta = -2, values beyond the clipped ends clamp to 0 and 15
    v = np.linspace(-4.0, 4.0, 33, dtype=np.float32)[None, :]
    q, a, b = quant.quant_asym(v, clip=0.5)
    assert b[0] == np.float32(-2.0) and a[0] == np.float32(np.float32(4.0) / np.float32(15.0))
    assert np.all(q[0, v[0] <= -2.0] == 0) and np.all(q[0, v[0] >= 2.0] == 15)
    inside = (v[0] > -2.0) & (v[0] < 2.0)
    err = np.abs(quant.dequant(q, a, b)[0, inside] - v[0, inside])
    assert np.all(err <= a[0] * 0.5 * (1 + 1e-6))
    q1, a1, b1 = quant.quant_asym(v, clip=1.0)
    q0, a0, b0 = quant.quant_asym(v)
    assert np.array_equal(q1, q0) and np.array_equal(a1, a0)


def test_asym_fp16_params_exact_case_equals_fp32():
    # range 7.5 over 15 levels: alpha = 0.5 and beta = -3.5 are fp16 numbers, so storing the
    # parameters in fp16 changes nothing: same codes, same values
    rng = np.random.default_rng(5)
    v = np.concatenate([[-3.5, 4.0], rng.uniform(-3.5, 4.0, 62)]).astype(np.float32)[None]
    q32, a32, b32 = quant.quant_asym(v)
    q16, a16, b16 = quant.quant_asym(v, param_fp16=True)
    assert a16.dtype == np.float16 and b16.dtype == np.float16
    assert a16[0] == np.float16(0.5) and b16[0] == np.float16(-3.5)
    np.testing.assert_array_equal(q16, q32)
    np.testing.assert_array_equal(a16.astype(np.float32), a32)
    np.testing.assert_array_equal(b16.astype(np.float32), b32)


@pytest.mark.parametrize("bits", [4, 8])
def test_asym_fp16_params_nearest_stored_level(bits):
    # with fp16 parameters every code is the nearest level a16 c + b16 of what is stored
    # (brute force over all 2^N levels; exact ties within 1e-3 of a step may go either way)
    rng = np.random.default_rng(6 + bits)
    v = (rng.standard_normal((50, 128)) * rng.uniform(0.01, 300, (50, 1))).astype(np.float32)
    q, a16, b16 = quant.quant_asym(v, bits=bits, param_fp16=True)
    a16, b16 = a16.reshape(-1), b16.reshape(-1)
    levels = np.arange(2 ** bits, dtype=np.float64)
    deq_all = a16.astype(np.float64)[:, None, None] * levels[None, None, :] + b16.astype(np.float64)[:, None, None]
    err_all = np.abs(deq_all - v.astype(np.float64)[:, :, None])
    best = err_all.min(axis=-1)
    mine = np.take_along_axis(err_all, q[:, :, None], axis=-1)[..., 0]
    assert np.all(mine <= best + 1e-3 * a16.astype(np.float64)[:, None])
    # and the stored pair is the fp32 pair rounded to nearest fp16
    _, a32, b32 = quant.quant_asym(v, bits=bits)
    np.testing.assert_array_equal(a16, a32.reshape(-1).astype(np.float16))
    np.testing.assert_array_equal(b16, b32.reshape(-1).astype(np.float16))


def test_asym_fp16_params_saturate_and_degenerate():
    # a range beyond fp16: alpha and beta saturate at 65504 instead of becoming inf
    v = np.array([[-1.0e6, 1.0e6, 0.0, 5.0e5]], np.float32)
    q, a16, b16 = quant.quant_asym(v, param_fp16=True)
    assert a16[0] == np.float16(65504) and b16[0] == np.float16(-65504)
    t = np.rint((v.astype(np.float64) + 65504.0) / 65504.0)
    np.testing.assert_array_equal(q, np.clip(t, 0, 15).astype(np.int64))
    # a constant group, and a range whose alpha underflows fp16 to 0: both constant
    for row in (np.full(16, 2.5, np.float32), np.linspace(1.0, 1.0 + 15 * 2e-8, 16).astype(np.float32)):
        q, a16, b16 = quant.quant_asym(row[None], param_fp16=True)
        assert a16[0] == np.float16(1.0) and np.all(q == 0)
        assert b16[0] == np.float16(row.min())
