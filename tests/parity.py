"""Comparison helpers for the GPU parity tests (test code; not part of the oracle).

Tolerances (per output row unless stated):
  * rotated values (fp32 accumulate vs the oracle's fp64):  |d| <= 1e-5 * max|row|
  * 4-bit codes from identical fp32 quantizer inputs:      bit-exact
  * 4-bit codes after a rotation: at most 1e-4 of the codes (and at least one may,
    whatever the size: an fp32-accumulated value within one rounding of a boundary can
    fall on either side) may differ, each by exactly one step, and each such element
    must sit on a rounding boundary in the oracle's own arithmetic (its scaled value
    (y - beta)/alpha within 1e-3 of k + 1/2, or the group's alpha/beta moved by the
    rotation's rounding); the same for 8-bit codes
  * scales alpha, beta after a rotation:                    relative 1e-5 (of the group range)
  * int32 accumulators from identical codes:                bit-exact
  * fp16 outputs from identical codes:                      |d| <= 2e-3 * max|row|
"""

import numpy as np

from oracle import quant


def unpack(p, signed):
    return quant.unpack_nibbles(np.asarray(p), signed=signed)


def assert_rot_close(gpu, ora, rel=1e-5):
    gpu = np.asarray(gpu, dtype=np.float64)
    ora = np.asarray(ora, dtype=np.float64)
    scale = np.abs(ora).max(axis=-1, keepdims=True)
    bad = np.abs(gpu - ora) > rel * scale
    assert not bad.any(), f"{bad.sum()} rotated values off by > {rel} x row max; worst " \
        f"{(np.abs(gpu - ora) / np.maximum(scale, 1e-30)).max():.3g}"


def assert_params_close(g_alpha, o_alpha, g_beta=None, o_beta=None, rel=1e-5):
    ga = np.asarray(g_alpha, dtype=np.float64)
    oa = np.asarray(o_alpha, dtype=np.float64)
    assert np.all(np.abs(ga - oa) <= rel * np.abs(oa)), "alpha differs"
    if g_beta is not None:
        gb = np.asarray(g_beta, dtype=np.float64)
        ob = np.asarray(o_beta, dtype=np.float64)
        # beta is a min: compare against the group's range (15 alpha)
        assert np.all(np.abs(gb - ob) <= rel * 15 * oa), "beta differs"


def code_flips(g_codes, o_codes, o_y32=None, o_alpha=None, o_beta=None, group=None,
               max_frac=1e-4, boundary_tol=1e-3):
    """Assert the codes agree up to the allowed rounding-boundary flips; return the count."""
    g = np.asarray(g_codes, dtype=np.int64)
    o = np.asarray(o_codes, dtype=np.int64)
    assert g.shape == o.shape
    d = g - o
    nflip = int(np.count_nonzero(d))
    assert np.all(np.abs(d) <= 1), f"a code differs by more than one step (max {np.abs(d).max()})"
    assert nflip <= max(1.0, max_frac * d.size), f"{nflip} flips in {d.size} codes exceeds {max_frac}"
    if nflip and o_y32 is not None:
        K = o.shape[-1]
        group = K if group is None else group
        a = np.repeat(np.asarray(o_alpha, dtype=np.float64).reshape(*o.shape[:-1], -1), group, axis=-1)
        b = np.repeat(np.asarray(o_beta, dtype=np.float64).reshape(*o.shape[:-1], -1), group, axis=-1)
        t = (np.asarray(o_y32, dtype=np.float64) - b) / a
        frac = np.abs(t - np.floor(t) - 0.5)
        idx = np.nonzero(d)
        assert np.all(frac[idx] <= boundary_tol), "a code flip is not at a rounding boundary"
    return nflip


def assert_out_close(gpu, ora, rel=2e-3):
    gpu = np.asarray(gpu, dtype=np.float64)
    ora = np.asarray(ora, dtype=np.float64)
    scale = np.abs(ora).max(axis=-1, keepdims=True)
    err = np.abs(gpu - ora)
    assert np.all(err <= rel * scale), f"output off by {(err / np.maximum(scale, 1e-30)).max():.3g} x row max"
