"""GPU parity: the HIP path (through the C ABI) against the CPU oracle, element by
element on the same seeded inputs.  Tolerances are documented in tests/parity.py."""

import numpy as np
import pytest
import torch

from oracle import hadamard as ohad
from oracle import kv as okv
from oracle import linear as olin
from oracle import quant as oq
from oracle import rotate as orot
from paper_2405_16406_amd import sq, workloads

import parity

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def say(msg):
    print(f"[gpu case] {msg}", flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def had_table(a):
    """Oracle's dense factor (the paper allows any Hadamard matrix), uploaded."""
    return None if a == 1 else dev(ohad.dense_factor(a))


def check_act(x, a, b, group=None, sample_rows=None, max_frac=1e-4):
    """GPU sq_had_quant_act vs oracle.had_quant_act on fp16 rows x."""
    K = x.shape[1]
    group = K if group is None else group
    ha = None if a == 1 else ohad.dense_factor(a)
    q, al, be, rot = sq.had_quant_act(dev(x), had_table(a), b, group=group, dbg=True)
    gq, gal, gbe, grot = host(q), host(al), host(be), host(rot)
    rows = np.arange(x.shape[0]) if sample_rows is None else sample_rows
    xs = x[rows]
    op, oal, obe, oy, oc = olin.had_quant_act(xs, ha, b, group=group)
    gc = parity.unpack(gq[rows], signed=False)
    if a * b == 1:
        np.testing.assert_array_equal(grot[rows], oy)
        np.testing.assert_array_equal(gq[rows], op)
        np.testing.assert_array_equal(gal[rows], oal)
        np.testing.assert_array_equal(gbe[rows], obe)
        return 0
    parity.assert_rot_close(grot[rows], oy)
    parity.assert_params_close(gal[rows], oal, gbe[rows], obe)
    return parity.code_flips(gc, oc, oy, oal, obe, group, max_frac=max_frac)


# ---------------------------------------------------------------- activations

def check_act8(x, a, b, group=None):
    """sq_had_quant_act with bits = 8 vs the oracle: one code per byte."""
    K = x.shape[1]
    group = K if group is None else group
    ha = None if a == 1 else ohad.dense_factor(a)
    q, al, be, rot = sq.had_quant_act(dev(x), had_table(a), b, group=group, bits=8, dbg=True)
    gq, gal, gbe, grot = host(q), host(al), host(be), host(rot)
    op, oal, obe, oy, oc = olin.had_quant_act(x, ha, b, bits=8, group=group)
    assert gq.shape == (x.shape[0], K)
    if a * b == 1:
        np.testing.assert_array_equal(gq, op)
        np.testing.assert_array_equal(gal, oal)
        np.testing.assert_array_equal(gbe, obe)
        return 0
    parity.assert_rot_close(grot, oy)
    parity.assert_params_close(gal, oal, gbe, obe)
    return parity.code_flips(gq.astype(np.int64), oc, oy, oal, obe, group)


@pytest.mark.parametrize("K", [8, 4096, 4104, 16392])
def test_identity_quant_8bit_bit_exact(K):
    say(f"had_quant_act 8-bit identity K={K}")
    x = workloads.outlier_acts(workloads.rng_for(K + 8), 5, K, max(1, K // 100), 50.0)
    assert check_act8(x, 1, 1) == 0


@pytest.mark.parametrize("a,b,M,group", [(1, 256, 16, None), (28, 512, 6, None), (172, 64, 3, None), (28, 16, 9, 224)])
def test_rotated_quant_8bit(a, b, M, group):
    say(f"had_quant_act 8-bit a={a} b={b} M={M} group={group}")
    x = workloads.outlier_acts(workloads.rng_for(a + b + M + 80), M, a * b, max(1, a * b // 100), 50.0)
    check_act8(x, a, b, group)


def check_act_var(x, a, b, bits=4, group=None, clip=1.0, signs=None, h_gpu=None, s_gpu=None, sample_rows=None):
    """sq_had_quant_act_ex (clip ratio, random-sign Hadamard S H) vs the oracle.  h_gpu and
    s_gpu replace the uploads of H_a and signs (views at other alignments); sample_rows: the
    GPU quantizes every row, the oracle those rows."""
    K = x.shape[1]
    group = K if group is None else group
    ha = None if a == 1 else ohad.dense_factor(a)
    if s_gpu is None and signs is not None:
        s_gpu = dev(signs.astype(np.int8))
    q, al, be, rot = sq.had_quant_act(dev(x), had_table(a) if h_gpu is None else h_gpu, b, group=group, bits=bits,
                                      dbg=True, clip=clip, signs=s_gpu)
    gq, gal, gbe, grot = host(q), host(al), host(be), host(rot)
    if sample_rows is not None:
        x, gq, gal, gbe, grot = x[sample_rows], gq[sample_rows], gal[sample_rows], gbe[sample_rows], grot[sample_rows]
    op, oal, obe, oy, oc = olin.had_quant_act(x, ha, b, bits=bits, group=group, clip=clip, signs=signs)
    gc = parity.unpack(gq, signed=False) if bits == 4 else gq.astype(np.int64)
    if a * b == 1:
        np.testing.assert_array_equal(grot, oy)
        np.testing.assert_array_equal(gq, op)
        np.testing.assert_array_equal(gal, oal)
        np.testing.assert_array_equal(gbe, obe)
        return 0
    parity.assert_rot_close(grot, oy)
    parity.assert_params_close(gal, oal, gbe, obe)
    return parity.code_flips(gc, oc, oy, oal, obe, group)


def rand_signs(n, seed):
    return np.where(workloads.rng_for(seed).random(n) < 0.5, -1, 1).astype(np.int8)


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("K", [8, 4096, 16392])
def test_identity_quant_clipped_bit_exact(bits, K):
    # the unrotated per-token kernel with a clipped range; and S alone (n = 1) on the generic one
    say(f"had_quant_act_ex identity {bits}-bit K={K} clip 0.9 / 0.95, signs [-1]")
    x = workloads.outlier_acts(workloads.rng_for(K + 90), 5, K, max(1, K // 100), 50.0)
    assert check_act_var(x, 1, 1, bits, clip=0.9) == 0
    assert check_act_var(x, 1, 1, bits, clip=0.95) == 0
    assert check_act_var(x, 1, 1, bits, signs=np.array([-1], np.int8), clip=0.95) == 0


# R4 shapes on the matrix-core kernels (pair: 172 x 64; lines: 28 x 512, 28 x 1024), a
# Sylvester-only and a per-group case on the generic kernel; signs, clip, or both
VAR_SHAPES = [(172, 64, 5, None), (28, 512, 4, None), (28, 1024, 3, None), (1, 256, 6, None), (28, 16, 5, 224)]


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("a,b,M,group", VAR_SHAPES)
def test_rotated_quant_variants(a, b, M, group, bits):
    say(f"had_quant_act_ex {bits}-bit a={a} b={b} M={M} group={group}: signs, clip 0.9, both")
    n = a * b
    x = workloads.outlier_acts(workloads.rng_for(a + b + M + 91), M, 2 * n if n < 1024 else n,
                               max(1, n // 100), 50.0)
    s = rand_signs(n, a + b)
    check_act_var(x, a, b, bits, group, signs=s)
    check_act_var(x, a, b, bits, group, clip=0.9)
    check_act_var(x, a, b, bits, group, clip=0.95, signs=s)
    # all-plus signs are the plain rotation: the same codes as sq_had_quant_act
    plain = [host(t) for t in sq.had_quant_act(dev(x), had_table(a), b, group=group, bits=bits)[:3]]
    ones = [host(t) for t in sq.had_quant_act(dev(x), had_table(a), b, group=group, bits=bits,
                                              signs=dev(np.ones(n, np.int8)))[:3]]
    for u, v in zip(plain, ones):
        np.testing.assert_array_equal(u, v)


@pytest.mark.parametrize("bits", [4, 8])
def test_rotated_quant_variants_full(bits):
    # the matrix-core kernels' variant instantiations at the full R4 sizes (every row on the
    # GPU, sampled rows against the oracle): LLaMA-2-7B [2048, 11008] (pair kernel) and
    # LLaMA-3-8B [4096, 14336] (line kernel), random signs with clip 0.9
    for shape, a, rows in ((workloads.LLAMA2_7B_MLP, 172, [0, 1, 2, 3, 1023, 2044, 2047]),
                           (workloads.LLAMA3_8B_MLP, 28, [0, 5, 2048, 4095])):
        say(f"had_quant_act_ex {bits}-bit {shape.name}: signs + clip 0.9, sampled rows")
        x = workloads.mlp_inputs(shape)["x_down"]
        s = rand_signs(shape.inter, 96 + a)
        check_act_var(x, a, shape.had_pow2, bits, signs=s, clip=0.9, sample_rows=np.array(rows))


def test_rotated_quant_variants_other_layouts():
    # an H_a or an S that is not 16- resp. 8-byte aligned leaves the matrix-core kernels for
    # the generic one; the results still follow the oracle
    say("had_quant_act_ex 172x64: H at +1 byte, signs at +1 byte")
    a, b, M = 172, 64, 4
    n = a * b
    x = workloads.outlier_acts(workloads.rng_for(92), M, n, n // 100, 50.0)
    hbuf = dev(np.concatenate([[0], ohad.dense_factor(a).reshape(-1)]).astype(np.int8))
    hg = hbuf[1:].view(a, a)
    s = rand_signs(n, 93)
    sbuf = dev(np.concatenate([[1], s]).astype(np.int8))
    check_act_var(x, a, b, 4, h_gpu=hg, signs=s, clip=0.9)
    check_act_var(x, a, b, 4, signs=s, s_gpu=sbuf[1:], clip=0.95)
    check_act_var(x, a, b, 8, signs=s, s_gpu=sbuf[1:])


def test_pack_w4_random_sign_chain():
    # the random Hadamard R = S H folded into the weights and applied to the activations
    # with the same S: the product keeps x W^T (Sec. 2.2; rotation invariance of Sec. 3.1)
    say("pack_w4_ex + had_quant_act_ex (signs) -> w4a4_linear, 28 x 32")
    a, b = 28, 32
    n = a * b
    rng = workloads.rng_for(94)
    w = workloads.weights(rng, 64, n)
    x = workloads.outlier_acts(rng, 16, n, 8, 20.0)
    s = rand_signs(n, 95)
    sg = dev(s)
    wq, wa, rs = sq.pack_w4(dev(w), had_table(a), b, signs=sg)
    owp, owa, ors, oqw = olin.pack_w4(w, ohad.dense_factor(a), b, signs=s)
    gqw = parity.unpack(host(wq), signed=True)
    np.testing.assert_array_equal(host(rs), gqw.sum(1))
    parity.assert_params_close(host(wa), owa)
    parity.code_flips(gqw, oqw)
    q, al, be, _ = sq.had_quant_act(dev(x), had_table(a), b, signs=sg)
    y, acc = sq.w4a4_linear(q, al, be, wq, wa, rs, dbg=True)
    # the GPU's own codes through the exact product
    oy, oacc = olin.w4a4_linear(parity.unpack(host(q), signed=False), host(al)[:, 0], host(be)[:, 0], gqw,
                                host(wa), host(rs))
    np.testing.assert_array_equal(host(acc), oacc)
    parity.assert_out_close(host(y), oy)
    # and the result approximates x W^T as the plain rotation does (4-bit error bound)
    ref = x.astype(np.float64) @ w.astype(np.float64).T
    err = np.abs(host(y).astype(np.float64) - ref).max() / np.abs(ref).max()
    assert err < 0.25, err


def test_tiny_identity_quant_bit_exact():
    say("had_quant_act tiny identity")
    x, _ = workloads.tiny_inputs()
    assert check_act(x, 1, 1) == 0


@pytest.mark.parametrize("K", [8, 4096, 4104, 8192, 8200, 16384, 16392, 32768])
def test_identity_quant_row_lengths(K):
    # each row-length range has its own chunks-per-thread instantiation
    say(f"had_quant_act identity K={K}")
    rng = workloads.rng_for(K)
    x = workloads.outlier_acts(rng, 5, K, max(1, K // 100), 50.0)
    assert check_act(x, 1, 1) == 0


def test_tiny_sylvester256():
    say("had_quant_act tiny Sylvester 256")
    x, _ = workloads.tiny_inputs()
    check_act(x, 1, 256)


@pytest.mark.parametrize("a,b,M", [(28, 4, 37), (172, 2, 5), (28, 16, 64), (1, 64, 3), (1, 1024, 2),
                                   (172, 64, 9), (28, 512, 4), (28, 1024, 3)])
def test_kronecker_shapes_small(a, b, M):
    say(f"had_quant_act a={a} b={b} M={M}")
    rng = workloads.rng_for(100 + a + b + M)
    x = workloads.outlier_acts(rng, M, a * b, max(1, a * b // 100), 50.0)
    check_act(x, a, b)


def test_blockwise_rotation_and_groups():
    say("had_quant_act block rotation n<K with group 128")
    rng = workloads.rng_for(7)
    x = workloads.outlier_acts(rng, 19, 28 * 8 * 4, 6, 50.0)
    check_act(x, 28, 8, group=224)
    check_act(x, 1, 1, group=128)


def test_edge_rows():
    say("had_quant_act edge rows")
    K = 28 * 64
    x = np.zeros((8, K), dtype=np.float16)
    x[1, :] = 0.5                     # constant row
    x[2, 17] = 300.0                  # single outlier
    x[3, :] = np.float16(-65504.0)    # fp16 extreme, constant
    x[4, ::2] = 1.0
    x[5] = workloads.outlier_acts(workloads.rng_for(3), 1, K, 3, 50.0)[0]
    x[6, 40] = np.float16(6e-8)       # smallest fp16 subnormal, alone
    x[7, ::3] = np.float16(-3e-6)     # subnormal values only
    check_act(x, 28, 64)
    check_act(x, 1, 1)


@pytest.mark.parametrize("a,b", [(28, 512), (172, 64), (28, 1024)])
def test_edge_rows_fast_paths(a, b):
    # the same degenerate rows through the MFMA kernels of the registered dense orders
    say(f"had_quant_act edge rows H{a} (x) S{b}")
    K = a * b
    x = np.zeros((9, K), dtype=np.float16)
    x[1, :] = 0.5
    x[2, 17] = 300.0
    x[3, :] = np.float16(-65504.0)
    x[4, ::2] = 1.0
    x[5] = workloads.outlier_acts(workloads.rng_for(4), 1, K, 3, 50.0)[0]
    x[6, 40] = np.float16(6e-8)
    x[7, ::3] = np.float16(-3e-6)
    x[8, K - 1] = -2.0                # last element only
    # Structured rows rotate to a few distinct values; e.g. a row whose rotation is mostly
    # zeros between symmetric extremes puts all those zeros exactly on the 7.5 boundary,
    # where the kernels (one fma, unscaled domain) and eq. 1 step by step may round apart.
    # No cap on the count, but every differing code must still sit on a rounding boundary.
    nflip = check_act(x, a, b, max_frac=1.0)
    say(f"  {nflip} boundary ties rounded the other way")


def test_llama2_7b_act_full():
    say("had_quant_act LLaMA-2-7B M=2048: identity [2048,4096] and R4 H172xH64 [2048,11008]")
    inp = workloads.mlp_inputs(workloads.LLAMA2_7B_MLP)
    assert check_act(inp["x_in"], 1, 1) == 0
    check_act(inp["x_down"], 172, 64)


def test_llama3_8b_act_full():
    say("had_quant_act LLaMA-3-8B M=4096: R4 H28xH512 [4096,14336]")
    inp = workloads.mlp_inputs(workloads.LLAMA3_8B_MLP)
    check_act(inp["x_down"], 28, 512)


def test_llama2_70b_decode_act():
    for shape in workloads.LLAMA2_70B_DECODE:
        say(f"had_quant_act {shape.name}: R4 H28xH1024 [M,28672]")
        inp = workloads.mlp_inputs(shape)
        assert check_act(inp["x_in"], 1, 1) == 0
        check_act(inp["x_down"], 28, 1024)


@pytest.mark.parametrize("a,b,M", [(172, 64, 1), (172, 64, 7), (172, 64, 1027), (28, 512, 3), (28, 512, 13)])
def test_kron_pair_partial_row_sets(a, b, M):
    say(f"had_quant_act H{a} (x) S{b}, M={M}: rows in sets of 4, last set partial")
    x = workloads.outlier_acts(workloads.rng_for(900 + M + a), M, a * b, a * b // 100, 50.0)
    check_act(x, a, b)


@pytest.mark.parametrize("a,b", [(172, 64), (28, 512)])
def test_kron_pair_strided_input_nan_padding(a, b):
    say(f"had_quant_act H{a} (x) S{b} on a strided input whose row padding is NaN")
    M, K = 9, a * b
    x = workloads.outlier_acts(workloads.rng_for(77), M, K, K // 100, 50.0)
    wide = np.full((M, K + 96), np.nan, dtype=np.float16)
    wide[:, :K] = x
    h = had_table(a)
    r1 = [host(v) for v in sq.had_quant_act(dev(wide)[:, :K], h, b)[:3]]
    r2 = [host(v) for v in sq.had_quant_act(dev(x), h, b)[:3]]
    for u, v in zip(r1, r2):
        np.testing.assert_array_equal(u, v)


@pytest.mark.parametrize("a,b", [(172, 64), (28, 512), (28, 1024)])
def test_kron_unaligned_factor_kernel(a, b):
    # an H_a that is not 16-byte aligned (plain 4-bit rotation, no variant) takes the
    # register-prefetch kernel instead of the LDS-staged matrix-core kernels
    say(f"had_quant_act H{a} (x) S{b} with H_a at +1 byte: register-prefetch kernel")
    x = workloads.outlier_acts(workloads.rng_for(31), 37, a * b, a * b // 100, 50.0)
    hbuf = dev(np.concatenate([[0], ohad.dense_factor(a).reshape(-1)]).astype(np.int8))
    hg = hbuf[1:].view(a, a)
    assert hg.data_ptr() % 16 != 0
    ha = ohad.dense_factor(a)
    q, al, be, rot = sq.had_quant_act(dev(x), hg, b, dbg=True)
    gq, gal, gbe, grot = host(q), host(al), host(be), host(rot)
    op, oal, obe, oy, oc = olin.had_quant_act(x, ha, b)
    parity.assert_rot_close(grot, oy)
    parity.assert_params_close(gal, oal, gbe, obe)
    parity.code_flips(parity.unpack(gq, signed=False), oc, oy, oal, obe, a * b)


@pytest.mark.parametrize("a,b,M", [(28, 512, 33), (172, 64, 21), (28, 1024, 5)])
def test_debug_output_does_not_change_results(a, b, M):
    say(f"had_quant_act with and without dbg_rot a={a} b={b} M={M}")
    rng = workloads.rng_for(500 + a + M)
    x = dev(workloads.outlier_acts(rng, M, a * b, max(1, a * b // 100), 50.0))
    h = had_table(a)
    r1 = [host(v) for v in sq.had_quant_act(x, h, b, dbg=False)[:3]]
    r2 = [host(v) for v in sq.had_quant_act(x, h, b, dbg=True)[:3]]
    for u, v in zip(r1, r2):
        assert np.array_equal(u, v)


def test_deterministic():
    say("had_quant_act determinism")
    x = workloads.mlp_inputs(workloads.LLAMA2_7B_MLP, rows=64)["x_down"]
    t = dev(x)
    h = had_table(172)
    r1 = [host(v) for v in sq.had_quant_act(t, h, 64)[:3]]
    r2 = [host(v) for v in sq.had_quant_act(t, h, 64)[:3]]
    for u, v in zip(r1, r2):
        assert np.array_equal(u, v)


# ---------------------------------------------------------------- weights

def check_w(w, a, b):
    ha = None if a == 1 else ohad.dense_factor(a)
    wq, wa, rs = sq.pack_w4(dev(w), had_table(a), b)
    gq, gwa, grs = host(wq), host(wa), host(rs)
    op, owa, ors, oc = olin.pack_w4(w, ha, b)
    gc = parity.unpack(gq, signed=True)
    np.testing.assert_array_equal(grs, gc.sum(1))
    if a * b == 1:
        np.testing.assert_array_equal(gq, op)
        np.testing.assert_array_equal(gwa, owa)
        np.testing.assert_array_equal(grs, ors)
        return 0
    parity.assert_params_close(gwa, owa)
    w32 = orot.rotate_rows(w, ha, b).astype(np.float32)
    n = parity.code_flips(gc, oc)
    if n:
        # every flipped weight code sits on a rounding boundary of the oracle's own arithmetic
        t = w32.astype(np.float64) / owa.astype(np.float64)[:, None]
        frac = np.abs(t - np.floor(t) - 0.5)
        assert np.all(frac[np.nonzero(gc - oc)] <= 1e-3)
    return n


def test_pack_w4_tiny_and_kronecker():
    say("pack_w4 tiny (none / Sylvester 256) and small Kronecker")
    _, w = workloads.tiny_inputs()
    assert check_w(w, 1, 1) == 0
    check_w(w, 1, 256)
    rng = workloads.rng_for(11)
    check_w(workloads.weights(rng, 37, 28 * 32), 28, 32)
    check_w(workloads.weights(rng, 20, 172 * 4), 172, 4)
    z = np.zeros((3, 256), dtype=np.float16)
    assert check_w(z, 1, 1) == 0


def test_pack_w4_stacked_rows_equal_separate():
    say("pack_w4 of stacked gate/up rows equals the two packs stacked")
    rng = workloads.rng_for(12)
    w1, w2 = workloads.weights(rng, 64, 512), workloads.weights(rng, 40, 512)
    both = [host(t) for t in sq.pack_w4(dev(np.concatenate([w1, w2])))]
    a = [host(t) for t in sq.pack_w4(dev(w1))]
    b = [host(t) for t in sq.pack_w4(dev(w2))]
    for u, x, y in zip(both, a, b):
        np.testing.assert_array_equal(u, np.concatenate([x, y]))


def test_pack_w4_llama2_7b_down_full():
    say("pack_w4 LLaMA-2-7B down [4096,11008] folded with H172xH64")
    w = workloads.mlp_inputs(workloads.LLAMA2_7B_MLP, rows=1)["w_down"]
    check_w(w, 172, 64)


# ---------------------------------------------------------------- GEMM

def gemm_case(M, N, K, seed, bias=True, sample_rows=None):
    rng = workloads.rng_for(seed)
    qa = rng.integers(0, 16, size=(M, K))
    qw = rng.integers(-7, 8, size=(N, K))
    xa = rng.uniform(0.05, 3.0, M).astype(np.float32)
    xb = rng.uniform(-20.0, 0.0, M).astype(np.float32)
    wa = rng.uniform(1e-3, 2e-2, N).astype(np.float32)
    rs = qw.sum(1).astype(np.int32)
    bi = (rng.standard_normal(N) * 0.1).astype(np.float16) if bias else None
    args = (dev(oq.pack_nibbles(qa)), dev(xa), dev(xb), dev(oq.pack_nibbles(qw)), dev(wa), dev(rs),
            dev(bi) if bias else None)
    y, acc = sq.w4a4_linear(*args, dbg=True)      # element-wise epilogue with the raw accumulators
    gy, gacc = host(y), host(acc)
    rows = np.arange(M) if sample_rows is None else sample_rows
    oy, oacc = olin.w4a4_linear(qa[rows], xa[rows], xb[rows], qw, wa, rs, bi)
    np.testing.assert_array_equal(gacc[rows], oacc)
    parity.assert_out_close(gy[rows], oy)
    y_fast, _ = sq.w4a4_linear(*args)             # vector-store epilogue: same arithmetic
    np.testing.assert_array_equal(host(y_fast), gy)


@pytest.mark.parametrize("M,N,K", [(16, 256, 256), (37, 200, 320), (1, 8, 64), (130, 129, 128),
                                   (256, 384, 1024), (8, 1000, 512)])
def test_gemm_small_shapes(M, N, K):
    say(f"w4a4_linear M={M} N={N} K={K}")
    gemm_case(M, N, K, seed=M * 7 + N + K)


def test_gemm_extreme_codes():
    say("w4a4_linear extreme codes K=28672")
    M, N, K = 3, 64, 28672
    qa = np.full((M, K), 15)
    qw = np.full((N, K), -7)
    qw[1] = 7
    xa = np.ones(M, np.float32) * 1e-4
    xb = np.zeros(M, np.float32)
    wa = np.ones(N, np.float32) * 1e-2
    rs = qw.sum(1).astype(np.int32)
    y, acc = sq.w4a4_linear(dev(oq.pack_nibbles(qa)), dev(xa), dev(xb), dev(oq.pack_nibbles(qw)), dev(wa),
                            dev(rs), None, dbg=True)
    oy, oacc = olin.w4a4_linear(qa, xa, xb, qw, wa, rs)
    np.testing.assert_array_equal(host(acc), oacc)
    parity.assert_out_close(host(y), oy)


def test_gemm_llama2_7b_gate_sampled():
    say("w4a4_linear LLaMA-2-7B gate [2048x4096]x[11008x4096], sampled rows")
    rows = np.array([0, 1, 127, 128, 1000, 2047])
    gemm_case(2048, 11008, 4096, seed=21, bias=False, sample_rows=rows)


def test_gemm_llama3_8b_down_sampled():
    say("w4a4_linear LLaMA-3-8B down [4096x14336]x[4096x14336], sampled rows")
    rows = np.array([0, 255, 256, 4095])
    gemm_case(4096, 4096, 14336, seed=22, bias=False, sample_rows=rows)


def swiglu_case(M, I, K, seed, bias=True, ldh_pad=0, sample_rows=None):
    """GPU sq_w4a4_linear_swiglu vs oracle.swiglu_linear; gate/up weights interleaved on the
    device with interleave_gate_up (codes, scales, row sums and bias alike)."""
    rng = workloads.rng_for(seed)
    qa = rng.integers(0, 16, size=(M, K))
    qg, qu = rng.integers(-7, 8, size=(I, K)), rng.integers(-7, 8, size=(I, K))
    xa = rng.uniform(0.05, 3.0, M).astype(np.float32)
    xb = rng.uniform(-20.0, 0.0, M).astype(np.float32)
    # weight scales shrink with sqrt(K) so that g and u stay O(10) and SiLU(g) u within fp16
    ws = min(1.0, float(np.sqrt(256.0 / K)))
    ga = (rng.uniform(1e-3, 2e-2, I) * ws).astype(np.float32)
    ua = (rng.uniform(1e-3, 2e-2, I) * ws).astype(np.float32)
    rsg, rsu = qg.sum(1).astype(np.int32), qu.sum(1).astype(np.int32)
    bg = (rng.standard_normal(I) * 0.5).astype(np.float16) if bias else None
    bu = (rng.standard_normal(I) * 0.5).astype(np.float16) if bias else None
    il = sq.interleave_gate_up
    wq = il(dev(oq.pack_nibbles(qg)), dev(oq.pack_nibbles(qu))).contiguous()
    wa, rs = il(dev(ga), dev(ua)).contiguous(), il(dev(rsg), dev(rsu)).contiguous()
    bi = il(dev(bg), dev(bu)).contiguous() if bias else None
    full = torch.full((M, I + ldh_pad), float("nan"), dtype=torch.float16, device="cuda")
    h = sq.w4a4_linear_swiglu(dev(oq.pack_nibbles(qa)), dev(xa), dev(xb), wq, wa, rs, bias=bi, out=full[:, :I])
    torch.cuda.synchronize()
    rows = np.arange(M) if sample_rows is None else sample_rows
    oh, og, ou = olin.swiglu_linear(qa[rows], xa[rows], xb[rows], qg, ga, rsg, qu, ua, rsu, bg, bu)
    gh = host(h)[rows]
    assert np.isfinite(gh).all()
    parity.assert_out_close(gh, oh)
    if ldh_pad:
        assert torch.isnan(full[:, I:]).all(), "row padding of h was written"
    else:
        # rows 8 bytes off a 16-byte multiple take the element-wise stores: same arithmetic,
        # so the same bits as the staged whole-row stores
        odd = torch.full((M, I + 4), float("nan"), dtype=torch.float16, device="cuda")
        h2 = sq.w4a4_linear_swiglu(dev(oq.pack_nibbles(qa)), dev(xa), dev(xb), wq, wa, rs, bias=bi, out=odd[:, :I])
        np.testing.assert_array_equal(host(h2).view(np.uint16), host(h).view(np.uint16))
    return og


@pytest.mark.parametrize("M,I,K,bias,pad", [(1, 32, 64, False, 0), (7, 96, 128, True, 0), (16, 224, 320, True, 3),
                                            (17, 160, 256, True, 0), (33, 128, 128, False, 1),
                                            (130, 352, 512, True, 8), (300, 96, 320, True, 0)])
def test_swiglu_linear_shapes(M, I, K, bias, pad):
    # decode kernel (M <= 16), 128 x 128 tiles (M <= 128), 256 x 128 tiles; ragged M and N,
    # padded or odd output strides (element-wise stores)
    say(f"w4a4_linear_swiglu M={M} I={I} K={K} bias={bias} ldh pad {pad}")
    og = swiglu_case(M, I, K, seed=400 + M + I + K, bias=bias, ldh_pad=pad)
    if M * I >= 2000:  # the gate values reach SiLU's flat, curved and linear parts
        assert (og < -8).any() and (og > 8).any() and (np.abs(og) < 2).any()


def test_swiglu_linear_llama2_7b_sampled():
    say("w4a4_linear_swiglu LLaMA-2-7B gate+up [2048x4096]x[2x11008x4096], sampled rows")
    swiglu_case(2048, 11008, 4096, seed=41, bias=False, sample_rows=np.array([0, 1, 255, 256, 1500, 2047]))


def test_swiglu_linear_llama3_8b_sampled():
    say("w4a4_linear_swiglu LLaMA-3-8B gate+up [4096x4096]x[2x14336x4096], sampled rows")
    swiglu_case(4096, 14336, 4096, seed=42, bias=True, sample_rows=np.array([0, 4095]))


@pytest.mark.parametrize("M", [1, 8, 16])
def test_swiglu_linear_llama2_70b_decode(M):
    say(f"w4a4_linear_swiglu LLaMA-2-70B decode M={M}: [M,8192]x[2x28672,8192]")
    swiglu_case(M, 28672, 8192, seed=43 + M, bias=False)


@pytest.mark.parametrize("M", [1, 8, 16])
def test_gemm_llama2_70b_decode(M):
    say(f"w4a4_linear LLaMA-2-70B decode M={M}: [M,8192]x[28672,8192] and [M,28672]x[8192,28672]")
    gemm_case(M, 28672, 8192, seed=30 + M, bias=False)
    gemm_case(M, 8192, 28672, seed=40 + M, bias=False)


def test_gemm_decode_kernel():
    # M <= 16 runs the weight-streaming kernel: every M up to 16, ragged N (blocks of 16
    # rows; N picks 1 to 8 blocks per workgroup), K not a multiple of the 8 waves' 64-byte
    # steps, and K shorter than one step
    say("w4a4_linear decode kernel: M 1..16, ragged N and K, 1-8 row blocks per workgroup")
    for (M, N, K) in [(1, 8, 64), (2, 40, 128), (7, 1000, 4160), (16, 130, 3136), (11, 4097, 640),
                      (3, 8200, 256), (5, 12300, 192), (9, 16390, 128), (4, 20500, 64), (6, 24600, 128),
                      (16, 28672 + 48, 192), (13, 96, 28672)]:
        gemm_case(M, N, K, seed=M * 31 + N + K, bias=(M % 2 == 1))


def test_gemm_gemv_kernel():
    # M <= 2 runs the dot-product kernel: whole 1 KB chunks of a row per wave load, K/2 not
    # a multiple of 1 KB, K/2 shorter than one chunk, the largest K it takes (65536) and the
    # first it leaves to the 16-row kernel, fewer rows than waves, and runs of more than 64
    # rows per wave's share (more workgroups); M = 3 and 4 on 117 MB of weights, which it
    # also took before the streaming kernel did
    say("w4a4_linear dot-product decode kernel: M 1..4, ragged N and K")
    for (M, N, K) in [(1, 3, 64), (2, 8, 64), (1, 1000, 4160), (2, 4097, 2112), (1, 700, 65536),
                      (2, 300, 65600), (1, 2048 * 64 + 5, 64), (3, 8192, 28672), (4, 8197, 24576)]:
        gemm_case(M, N, K, seed=M * 37 + N + K, bias=(N % 2 == 1))


def test_gemm_stream_kernel():
    # 2 < M <= 16 on larger weights runs the LDS-streaming kernel (on a 256-CU part): ragged
    # N (a partial last block of 16 rows), K/2 not a multiple of the 256-byte stage, 1 to 16
    # blocks per workgroup, a single block, and runs of the 8 waves that cross one or two
    # block boundaries (16 blocks of 2 stages); rows past M of the 16-row blocks
    say("w4a4_linear LDS-streaming decode kernel: M 3..16, ragged N and K, runs across blocks")
    for (M, N, K) in [(16, 4096 * 3 + 40, 2112), (5, 16 * 256 * 16 - 16 * 7, 576), (3, 300, 65536),
                      (12, 8208, 2048), (8, 17, 16384), (16, 16, 8192), (7, 4096, 11008)]:
        gemm_case(M, N, K, seed=M * 41 + N + K, bias=(K % 3 == 0))


@pytest.mark.parametrize("M,I,K,bias", [(6, 4128, 2112, True), (9, 32, 4096, False), (11, 28672, 8256, True),
                                        (16, 11008, 4096, True)])
def test_swiglu_stream_kernel(M, I, K, bias):
    # the LDS-streaming kernel with SiLU: pairs of a gate and an up block of 16 rows, a
    # single group of four blocks in all, a last workgroup with fewer pairs (LLaMA-2-7B:
    # 688 pairs, 3 per workgroup), and runs crossing block boundaries (17 stages a block)
    say(f"w4a4_linear_swiglu LDS-streaming decode kernel M={M} I={I} K={K} bias={bias}")
    swiglu_case(M, I, K, seed=700 + M + I + K, bias=bias)


@pytest.mark.parametrize("M,I,K,bias", [(1, 96, 4160, True), (2, 32, 64, False), (1, 2048 * 64 + 32, 64, True),
                                        (2, 4128, 2112, True), (3, 14336, 8192, False)])
def test_swiglu_gemv_kernel(M, I, K, bias):
    say(f"w4a4_linear_swiglu dot-product decode kernel M={M} I={I} K={K} bias={bias}")
    swiglu_case(M, I, K, seed=600 + M + I + K, bias=bias)


# ---------------------------------------------------------------- W4A8

def gemm8_case(M, N, K, seed, bias=True, sample_rows=None):
    rng = workloads.rng_for(seed)
    qa = rng.integers(0, 256, size=(M, K))
    qw = rng.integers(-7, 8, size=(N, K))
    xa = rng.uniform(0.003, 0.2, M).astype(np.float32)
    xb = rng.uniform(-20.0, 0.0, M).astype(np.float32)
    wa = rng.uniform(1e-3, 2e-2, N).astype(np.float32)
    rs = qw.sum(1).astype(np.int32)
    bi = (rng.standard_normal(N) * 0.1).astype(np.float16) if bias else None
    args = (dev(qa.astype(np.uint8)), dev(xa), dev(xb), dev(oq.pack_nibbles(qw)), dev(wa), dev(rs),
            dev(bi) if bias else None)
    y, acc = sq.w4a8_linear(*args, dbg=True)
    rows = np.arange(M) if sample_rows is None else sample_rows
    oy, oacc = olin.w4a4_linear(qa[rows], xa[rows], xb[rows], qw, wa, rs, bi)
    np.testing.assert_array_equal(host(acc)[rows], oacc)
    parity.assert_out_close(host(y)[rows], oy)
    y2, _ = sq.w4a8_linear(*args)
    np.testing.assert_array_equal(host(y2), host(y))


@pytest.mark.parametrize("M,N,K", [(1, 8, 64), (37, 200, 320), (130, 129, 128), (256, 384, 1024), (8, 1000, 512),
                                   (300, 390, 448)])
def test_w4a8_gemm_small_shapes(M, N, K):
    say(f"w4a8_linear M={M} N={N} K={K}")
    gemm8_case(M, N, K, seed=M * 5 + N + K)


@pytest.mark.parametrize("M,N,K", [(1, 8, 64), (2, 40, 128), (7, 1000, 4160), (16, 130, 3136), (11, 4097, 640),
                                   (16, 28672, 8192), (1, 8192, 28672), (13, 96, 28672),
                                   (1, 1001, 4160), (1, 2048 * 64 + 5, 64), (2, 8192, 8192), (1, 700, 65536),
                                   (1, 64, 65600), (8, 8192, 28672), (3, 4096 * 3 + 40, 2112),
                                   (5, 16 * 256 * 16 - 16 * 7, 576), (8, 17, 16384), (4, 4096, 11008)])
def test_w4a8_decode_shapes(M, N, K):
    # M <= 16 with 8-bit activations: the dot-product kernel for one row (two from 32 MB of
    # weights; ragged N and K, K/2 shorter than 1 KB, long runs, the largest K it takes and
    # the first it leaves), the LDS-streaming kernel up to 8 rows (ragged N, K/2 not a
    # multiple of its 256-byte stage, 1 to 16 blocks per workgroup, runs across block
    # boundaries) and the 16-row kernel (1, 2 or 4 blocks of 16 rows) otherwise
    say(f"w4a8_linear decode M={M} N={N} K={K}")
    gemm8_case(M, N, K, seed=M * 13 + N + K, bias=(M % 2 == 1))


def test_w4a8_prefill_kernels():
    # the ring kernels with 8-bit A blocks (128 x 256 tiles; 256 x 256 tiles from 256 such
    # tiles on): ragged M and N, K not a multiple of a 128-k stage
    say("w4a8_linear prefill ring kernel")
    for (M, N, K) in [(300, 390, 448), (257, 600, 320), (129, 1000, 2112), (640, 520, 1024), (2048, 300, 256),
                      (4096, 4096, 128), (4000, 4100, 320)]:
        gemm8_case(M, N, K, seed=M + N + K + 7)


def test_w4a8_gemm_extreme_codes():
    # the largest int32 sums the kernel forms: 16 x (255 - 128) x 7 and 16 x (0 - 128) x (-7)
    # over K = 2^17
    say("w4a8_linear extreme codes K=2^17")
    M, N, K = 2, 64, 1 << 17
    qa = np.full((M, K), 255)
    qa[1] = 0
    qw = np.full((N, K), 7)
    qw[1::2] = -7
    xa = np.full(M, 1e-6, np.float32)
    xb = np.zeros(M, np.float32)
    wa = np.full(N, 1e-2, np.float32)
    rs = qw.sum(1).astype(np.int32)
    y, acc = sq.w4a8_linear(dev(qa.astype(np.uint8)), dev(xa), dev(xb), dev(oq.pack_nibbles(qw)), dev(wa), dev(rs),
                            None, dbg=True)
    oy, oacc = olin.w4a4_linear(qa, xa, xb, qw, wa, rs)
    np.testing.assert_array_equal(host(acc), oacc)
    parity.assert_out_close(host(y), oy)


def test_w4a8_gemm_llama_sampled():
    say("w4a8_linear LLaMA-2-7B gate [2048x4096]x[11008x4096] and down [2048x11008]x[4096x11008], sampled rows")
    rows = np.array([0, 127, 128, 2047])
    gemm8_case(2048, 11008, 4096, seed=51, bias=False, sample_rows=rows)
    gemm8_case(2048, 4096, 11008, seed=52, bias=False, sample_rows=rows)


def test_w4a8_rotated_chain():
    # fp16 rows -> rotated 8-bit codes -> W4A8 product, against the oracle's whole chain
    say("W4A8 chain: had_quant_act(bits=8, Sylvester 256) -> pack_w4 -> w4a8_linear")
    x, w = workloads.tiny_inputs()
    q, al, be, _ = sq.had_quant_act(dev(x), None, 256, bits=8)
    wq, wa, rs = sq.pack_w4(dev(w), None, 256)
    y, acc = sq.w4a8_linear(q, al, be, wq, wa, rs, dbg=True)
    op, oxa, oxb, oy_rot, oqa = olin.had_quant_act(x, None, 256, bits=8)
    owp, owa, ors, oqw = olin.pack_w4(w, None, 256)
    gqa = host(q).astype(np.int64)
    if np.array_equal(gqa, oqa) and np.array_equal(parity.unpack(host(wq), signed=True), oqw):
        oy, oacc = olin.w4a4_linear(oqa, oxa[:, 0], oxb[:, 0], oqw, owa, ors)
        np.testing.assert_array_equal(host(acc), oacc)
        parity.assert_out_close(host(y), oy)
    else:  # a rounding-boundary flip upstream: the product of the GPU's own codes must still match
        oy, oacc = olin.w4a4_linear(gqa, host(al)[:, 0], host(be)[:, 0], parity.unpack(host(wq), signed=True),
                                    host(wa), host(rs))
        np.testing.assert_array_equal(host(acc), oacc)


# ---------------------------------------------------------------- decode attention

def attn_case(B, S, H, seed, scale=None, qscale=2.0, split=False):
    """GPU sq_attn_decode_kv4 (split: sq_attn_decode_kv4_split) vs oracle.attn_decode on a
    random 4-bit cache."""
    rng = workloads.rng_for(seed)
    kc, vc = rng.integers(0, 16, (B, S, H, 128)), rng.integers(0, 16, (B, S, H, 128))
    ka, va = (rng.uniform(0.01, 0.2, (B, S, H)).astype(np.float32) for _ in range(2))
    kb, vb = (rng.uniform(-1.5, 0.0, (B, S, H)).astype(np.float32) for _ in range(2))
    q = (rng.standard_normal((B, H, 128)) * qscale).astype(np.float16)
    kq, vq = oq.pack_nibbles(kc), oq.pack_nibbles(vc)
    fn = sq.attn_decode_kv4_split if split else sq.attn_decode_kv4
    out = fn(dev(q), dev(kq), dev(ka), dev(kb), dev(vq), dev(va), dev(vb), scale=scale)
    ref = okv.attn_decode(q, kq, ka, kb, vq, va, vb, scale)
    got = host(out)
    assert np.isfinite(got).all()
    parity.assert_out_close(got, ref)
    return got, ref, (va[..., None] * vc + vb[..., None])


@pytest.mark.parametrize("B,S,H", [(1, 1, 1), (1, 5, 3), (2, 17, 2), (3, 300, 5), (2, 1000, 8), (1, 129, 4),
                                   (2, 4099, 4)])
def test_attn_decode_shapes(B, S, H):
    # one token up to several thousand; ragged batches of 16; head counts that are and are
    # not a multiple of 8 (the XCD-aware head order applies to the former)
    say(f"attn_decode_kv4 B={B} S={S} H={H}")
    attn_case(B, S, H, seed=600 + B + S + H)


@pytest.mark.parametrize("split", [False, True])
def test_attn_decode_degenerate_scores(split):
    say(f"attn_decode_kv4 (split={split}): scale 0 (mean of V), a sharp softmax, a single token")
    got, ref, V = attn_case(2, 37, 3, seed=7, scale=0.0, split=split)
    parity.assert_out_close(got, V.mean(axis=1).astype(np.float16))
    attn_case(2, 200, 2, seed=8, scale=1.0, qscale=8.0, split=split)
    attn_case(1, 3000, 2, seed=10, scale=1.0, qscale=8.0, split=split)  # sharp, over many chunks
    got, ref, V = attn_case(1, 1, 4, seed=9, split=split)
    parity.assert_out_close(got, V[:, 0].astype(np.float16))


@pytest.mark.parametrize("B,S,H", [(1, 1, 1), (1, 5, 3), (2, 17, 2), (1, 129, 4), (1, 300, 5), (2, 4099, 4),
                                   (1, 1000, 33), (3, 777, 17), (1, 4096, 2), (1, 20000, 3), (8, 2048, 32)])
def test_attn_decode_split_shapes(B, S, H):
    # one chunk (the output written by the partial kernel) and many, up to the 64 the
    # combine takes; ragged chunks and batches; odd head counts (a wave's second head
    # missing) and counts below, at and past a 16-head group; the full [8, 2048, 32] cache
    nbytes = sq.attn_decode_workspace_bytes(B, S, H)
    say(f"attn_decode_kv4_split B={B} S={S} H={H} workspace {nbytes} bytes")
    attn_case(B, S, H, seed=640 + B + S + H, split=True)


def test_attn_decode_split_matches_unsplit():
    # the two kernels sum in different orders: their outputs agree to fp16 rounding
    say("attn_decode_kv4_split vs attn_decode_kv4 on the chain cache [2,1500,32,128]")
    q, k, v = (dev(t) for t in workloads.kv_inputs(B=2, S=1500, H=32, D=128))
    o = sq.qk_had_kvquant(q, k, v)
    qr = o["q_rot"][:, -1].contiguous()
    cache = (o["k_q"], o["k_alpha"], o["k_beta"], o["v_q"], o["v_alpha"], o["v_beta"])
    a = host(sq.attn_decode_kv4(qr, *cache)).astype(np.float32)
    b = host(sq.attn_decode_kv4_split(qr, *cache)).astype(np.float32)
    np.testing.assert_allclose(b, a, rtol=4e-3, atol=2e-3 * np.abs(a).max())


def test_attn_decode_split_workspace_checks():
    say("attn_decode_kv4_split: workspace too small, misaligned, overlapping, NULL")
    B, S, H = 1, 1000, 8
    rng = workloads.rng_for(650)
    kq, vq = (dev(rng.integers(0, 256, (B, S, H, 64), dtype=np.uint8)) for _ in range(2))
    ka, kb, va, vb = (dev(rng.uniform(0.01, 0.2, (B, S, H)).astype(np.float32)) for _ in range(4))
    q = dev(rng.standard_normal((B, H, 128)).astype(np.float16))
    need = sq.attn_decode_workspace_bytes(B, S, H)
    assert need > 0 and need % 528 == 0
    args = (q, kq, ka, kb, vq, va, vb)
    with pytest.raises(sq.SqError, match="SQ_ERR_SHAPE"):
        sq.attn_decode_kv4_split(*args, workspace=torch.empty(need - 16, dtype=torch.uint8, device="cuda"))
    big = torch.empty(need + 64, dtype=torch.uint8, device="cuda")
    with pytest.raises(sq.SqError, match="SQ_ERR_ALIGN"):
        sq.attn_decode_kv4_split(*args, workspace=big[4:need + 4])
    with pytest.raises(sq.SqError, match="SQ_ERR_ALIAS"):
        sq.attn_decode_kv4_split(*args, out=big[:B * H * 256].view(torch.float16).view(B, H, 128), workspace=big)
    L = sq.lib()
    st = L.sq_attn_decode_kv4_split(q.data_ptr(), kq.data_ptr(), ka.data_ptr(), kb.data_ptr(), vq.data_ptr(),
                                    va.data_ptr(), vb.data_ptr(), B, S, H, 128, 0.1, 32,
                                    torch.empty_like(q).data_ptr(), None, 0, None)
    assert st == sq.SQ_ERR_SHAPE
    # exactly the bytes asked for, and a B == 0 no-op with no workspace
    out = sq.attn_decode_kv4_split(*args, workspace=torch.empty(need, dtype=torch.uint8, device="cuda"))
    parity.assert_out_close(host(out), okv.attn_decode(*(host(t) for t in args)))
    e = torch.empty_like(q)
    assert L.sq_attn_decode_kv4_split(q.data_ptr(), kq.data_ptr(), ka.data_ptr(), kb.data_ptr(), vq.data_ptr(),
                                      va.data_ptr(), vb.data_ptr(), 0, S, H, 128, 0.1, 32, e.data_ptr(), None, 0,
                                      None) == sq.SQ_OK


def test_attn_decode_after_kv_quant_full():
    # the whole consumer chain at [8, 2048, 32, 128]: R3 + KV4 on the GPU, then the last
    # token's rotated query attends over the cache the GPU wrote; oracle on two batches
    say("qk_had_kvquant -> attn_decode_kv4 and _split [8, 2048, 32, 128], last token's query")
    q, k, v = workloads.kv_inputs()
    o = sq.qk_had_kvquant(dev(q), dev(k), dev(v))
    qr = o["q_rot"][:, -1].contiguous()
    cache = (o["k_q"], o["k_alpha"], o["k_beta"], o["v_q"], o["v_alpha"], o["v_beta"])
    for fn in (sq.attn_decode_kv4, sq.attn_decode_kv4_split):
        got = host(fn(qr, *cache))
        for b in (0, 7):
            sl = slice(b, b + 1)
            ref = okv.attn_decode(host(qr)[sl], *(host(t)[sl] for t in cache))
            parity.assert_out_close(got[sl], ref)


# ---------------------------------------------------------------- chain

def test_tiny_rotated_linear_chain():
    say("tiny rotated W4A4 linear chain (had_quant_act -> pack_w4 -> w4a4_linear)")
    x, w = workloads.tiny_inputs()
    q, al, be, _ = sq.had_quant_act(dev(x), None, 256)
    wq, wa, rs = sq.pack_w4(dev(w), None, 256)
    y, acc = sq.w4a4_linear(q, al, be, wq, wa, rs, dbg=True)
    gy = host(y)
    ref = olin.rotated_linear(x, w, None, 256)
    gqa = parity.unpack(host(q), signed=False)
    gqw = parity.unpack(host(wq), signed=True)
    if np.array_equal(gqa, ref["qa"]) and np.array_equal(gqw, ref["qw"]):
        np.testing.assert_array_equal(host(acc), ref["acc"])
        parity.assert_out_close(gy, ref["y"])
    else:
        # flipped codes move an output by alpha_m * s_n per flip and k
        dqa = np.abs(gqa - ref["qa"]).astype(np.float64)
        dqw = np.abs(gqw - ref["qw"]).astype(np.float64)
        bound = (ref["x_alpha"][:, None] * (dqa @ np.abs(ref["qw"]).T) * ref["w_alpha"][None, :]
                 + (np.abs(ref["qa"]) * ref["x_alpha"][:, None] + np.abs(ref["x_beta"])[:, None]) @ dqw.T
                 * ref["w_alpha"][None, :])
        err = np.abs(gy.astype(np.float64) - ref["y"].astype(np.float64))
        scale = np.abs(ref["y"].astype(np.float64)).max(1, keepdims=True)
        assert np.all(err <= 2e-3 * scale + 1.01 * bound)


# ---------------------------------------------------------------- KV

def check_kv(q, k, v, sample=None, bits=4, k_clip=1.0, v_clip=1.0):
    out = sq.qk_had_kvquant(dev(q), dev(k), dev(v), dbg=True, bits=bits, k_clip=k_clip, v_clip=v_clip)
    g = {n: host(t) for n, t in out.items() if t is not None}
    B, S, H, D = q.shape
    flat = lambda a: a.reshape(B * S * H, -1)
    idx = np.arange(B * S * H) if sample is None else sample
    qs, ks, vs = (flat(t)[idx][None, :, None, :] for t in (q, k, v))
    o = okv.qk_had_kvquant(qs, ks, vs, bits=bits, k_clip=k_clip, v_clip=v_clip)
    sel = lambda a: flat(a)[idx][None, :, None, :]
    codes = (lambda a: parity.unpack(a, False)) if bits == 4 else (lambda a: a.astype(np.int64))
    # Q R: fp16 of an fp32 sum vs fp16 of the fp64 value: one fp16 ulp of rounding plus the
    # 1e-5 x row-max allowance of an fp32-accumulated rotation (matters for values near 0)
    gq = sel(g["q_rot"]).astype(np.float64)
    oq_ = o["q_rot"].astype(np.float64)
    ulp = np.spacing(np.abs(o["q_rot"]).astype(np.float16)).astype(np.float64)
    rowmax = np.abs(oq_).max(axis=-1, keepdims=True)
    assert np.all(np.abs(gq - oq_) <= ulp + 1e-5 * rowmax)
    parity.assert_rot_close(sel(g["k_rot"]).reshape(-1, 128), o["k_rot"].reshape(-1, 128))
    parity.assert_params_close(sel(g["k_alpha"]), o["k_alpha"], sel(g["k_beta"]), o["k_beta"])
    parity.code_flips(codes(sel(g["k_q"])).reshape(-1, 128), o["k_codes"].reshape(-1, 128),
                      o["k_rot"].reshape(-1, 128), o["k_alpha"].reshape(-1, 1), o["k_beta"].reshape(-1, 1))
    np.testing.assert_array_equal(sel(g["v_q"]), o["v_q"])
    np.testing.assert_array_equal(sel(g["v_alpha"]), o["v_alpha"])
    np.testing.assert_array_equal(sel(g["v_beta"]), o["v_beta"])


def test_kv_small():
    say("qk_had_kvquant small [2,16,4,128] and ragged [1,3,5,128]")
    check_kv(*workloads.kv_inputs(B=2, S=16, H=4, D=128))
    check_kv(*workloads.kv_inputs(B=1, S=3, H=5, D=128))


@pytest.mark.parametrize("bits", [4, 8])
def test_kv_clipped(bits):
    # range clipping of the cache groups (0.95 is the cache ratio App. A compares against
    # unclipped min-max; 0.9 clips more); V codes stay bit-exact, K codes boundary-exact
    say(f"qk_had_kvquant_ex {bits}-bit, k_clip 0.9 / v_clip 0.95 and k_clip 0.95 / v_clip 1")
    q, k, v = workloads.kv_inputs(B=2, S=16, H=4, D=128)
    check_kv(q, k, v, bits=bits, k_clip=0.9, v_clip=0.95)
    check_kv(q, k, v, bits=bits, k_clip=0.95, v_clip=1.0)
    # clipping moves codes: the outermost values of a group take the end codes 0 and L
    out = sq.qk_had_kvquant(dev(q), dev(k), dev(v), bits=bits, k_clip=1.0, v_clip=0.5)
    vc = host(out["v_q"])
    vc = parity.unpack(vc, False) if bits == 4 else vc.astype(np.int64)
    L = 2 ** bits - 1
    assert np.all(vc.max(-1) == L) and np.all(vc.min(-1) == 0)


@pytest.mark.parametrize("bits", [4, 8])
def test_kv_fp16_params(bits):
    # fp16 group parameters: V bit-exact (parameters and codes); K parameters within one fp16
    # step of the oracle's (the rotation's fp32 rounding can tip the fp16 rounding), and K
    # codes those of the oracle's quantizer applied with the GPU's own stored pair
    say(f"qk_had_kvquant_ex {bits}-bit fp16 parameters [2,16,4,128] and [1,3,5,128], v_clip 0.95")
    for shape in ((2, 16, 4, 128), (1, 3, 5, 128)):
        q, k, v = workloads.kv_inputs(*shape)
        out = sq.qk_had_kvquant(dev(q), dev(k), dev(v), dbg=True, bits=bits, v_clip=0.95,
                                param_dtype=torch.float16)
        g = {n: host(t) for n, t in out.items() if t is not None}
        o = okv.qk_had_kvquant(q, k, v, bits=bits, v_clip=0.95, param_fp16=True)
        for nm in ("k_alpha", "k_beta", "v_alpha", "v_beta"):
            assert g[nm].dtype == np.float16
        np.testing.assert_array_equal(g["v_q"], o["v_q"])
        np.testing.assert_array_equal(g["v_alpha"], o["v_alpha"])
        np.testing.assert_array_equal(g["v_beta"], o["v_beta"])
        for nm in ("k_alpha", "k_beta"):
            gg, oo = g[nm].astype(np.float64), o[nm].astype(np.float64)
            assert np.all(np.abs(gg - oo) <= np.spacing(np.abs(o[nm])).astype(np.float64)), nm
        codes = (lambda a: parity.unpack(a, False)) if bits == 4 else (lambda a: a.astype(np.int64))
        kr = o["k_rot"].reshape(-1, 128)
        ka, kb = g["k_alpha"].reshape(-1, 1), g["k_beta"].reshape(-1, 1)
        parity.code_flips(codes(g["k_q"]).reshape(-1, 128), oq.asym_codes(kr, ka, kb, bits), kr,
                          ka.astype(np.float32), kb.astype(np.float32))


def test_attn_decode_fp16_params():
    # the consumer reads fp16 parameters: a random cache with fp16 parameters against the
    # oracle, and the whole chain from fp16-parameter KV quantization
    say("attn_decode_kv4_ex fp16 parameters: random cache [2,300,5], chain [1,257,4]")
    rng = workloads.rng_for(700)
    B, S, H = 2, 300, 5
    kc, vc = rng.integers(0, 16, (B, S, H, 128)), rng.integers(0, 16, (B, S, H, 128))
    ka, va = (rng.uniform(0.01, 0.2, (B, S, H)).astype(np.float16) for _ in range(2))
    kb, vb = (rng.uniform(-1.5, 0.0, (B, S, H)).astype(np.float16) for _ in range(2))
    q = (rng.standard_normal((B, H, 128)) * 2).astype(np.float16)
    kq, vq = oq.pack_nibbles(kc), oq.pack_nibbles(vc)
    for fn in (sq.attn_decode_kv4, sq.attn_decode_kv4_split):
        out = fn(dev(q), dev(kq), dev(ka), dev(kb), dev(vq), dev(va), dev(vb))
        parity.assert_out_close(host(out), okv.attn_decode(q, kq, ka, kb, vq, va, vb))
    qh, kh, vh = workloads.kv_inputs(1, 257, 4, 128)
    o = sq.qk_had_kvquant(dev(qh), dev(kh), dev(vh), param_dtype=torch.float16)
    qr = o["q_rot"][:, -1].contiguous()
    cache = [o[n] for n in ("k_q", "k_alpha", "k_beta", "v_q", "v_alpha", "v_beta")]
    for fn in (sq.attn_decode_kv4, sq.attn_decode_kv4_split):
        got = host(fn(qr, *cache))
        parity.assert_out_close(got, okv.attn_decode(host(qr), *[host(t) for t in cache]))


def test_kv8_small_and_sampled():
    # KV8: the same kernel storing one 8-bit code per byte
    say("qk_had_kvquant 8-bit [2,16,4,128], [1,3,5,128] and [8,2048,32,128] sampled")
    check_kv(*workloads.kv_inputs(B=2, S=16, H=4, D=128), bits=8)
    check_kv(*workloads.kv_inputs(B=1, S=3, H=5, D=128), bits=8)
    q, k, v = workloads.kv_inputs()
    rng = np.random.default_rng(1)
    sample = np.unique(np.concatenate([rng.choice(8 * 2048 * 32, 5000, replace=False), [0, 8 * 2048 * 32 - 1]]))
    check_kv(q, k, v, sample, bits=8)


def test_kv_full_sampled():
    say("qk_had_kvquant R3 KV [8,2048,32,128], sampled groups")
    q, k, v = workloads.kv_inputs()
    rng = np.random.default_rng(0)
    sample = np.unique(np.concatenate([rng.choice(8 * 2048 * 32, 20000, replace=False),
                                       [0, 8 * 2048 * 32 - 1]]))
    check_kv(q, k, v, sample)


# Each size class of the dispatch: 16 < M <= 128 (128 x 128 tiles, two K groups), fewer
# than 256 tiles of 256 x 256 (128 x 256 tiles of 8 waves), at least 256 such tiles
# (8-wave 256 x 256); ragged M, N and K (K % 128 == 64: a half stage)
GEMM_CLASS_SHAPES = [(64, 130, 192), (100, 1000, 2112), (300, 390, 448), (257, 257, 128), (520, 600, 320),
                     (384, 264, 2112), (4096, 4096, 192), (4000, 4100, 320)]


@pytest.mark.parametrize("M,N,K", GEMM_CLASS_SHAPES)
def test_gemm_size_classes(M, N, K):
    say(f"w4a4_linear M={M} N={N} K={K}: vector and element-wise stores")
    rng = workloads.rng_for(M + N + K)
    qa = rng.integers(0, 16, size=(M, K))
    qw = rng.integers(-7, 8, size=(N, K))
    xa = rng.uniform(0.05, 3.0, M).astype(np.float32)
    xb = rng.uniform(-20.0, 0.0, M).astype(np.float32)
    wa = rng.uniform(1e-3, 2e-2, N).astype(np.float32)
    rs = qw.sum(1).astype(np.int32)
    bi = (rng.standard_normal(N) * 0.1).astype(np.float16)
    args = (dev(oq.pack_nibbles(qa)), dev(xa), dev(xb), dev(oq.pack_nibbles(qw)), dev(wa), dev(rs), dev(bi))
    oy, oacc = olin.w4a4_linear(qa, xa, xb, qw, wa, rs, bi)
    y_dbg, acc = sq.w4a4_linear(*args, dbg=True)
    np.testing.assert_array_equal(host(acc), oacc)
    parity.assert_out_close(host(y_dbg), oy)
    y_fast, _ = sq.w4a4_linear(*args)                      # vector stores inside N
    np.testing.assert_array_equal(host(y_fast), host(y_dbg))
    wide = torch.zeros((M, N + 3), dtype=torch.float16, device=DEV)
    sq.w4a4_linear(*args, out=wide[:, :N])                 # odd ldy: element-wise stores
    np.testing.assert_array_equal(host(wide[:, :N]), host(y_dbg))
    assert not host(wide[:, N:]).any()
    w8 = (N + 1 + 7) // 8 * 8                              # ldy % 8 == 0: vector stores,
    wide8 = torch.zeros((M, w8), dtype=torch.float16, device=DEV)   # edge tiles element-wise
    sq.w4a4_linear(*args, out=wide8[:, :N])
    np.testing.assert_array_equal(host(wide8[:, :N]), host(y_dbg))
    assert not host(wide8[:, N:]).any()


# Operands of 2 GB and more do not fit the 31-bit buffer offsets of the ring and decode
# kernels, and take the register-staged kernels.  The big operand repeats a few seeded rows
# (built on the device), so the oracle computes the sampled outputs from those rows.  K % 128
# == 64 takes the half stage at the end of K.
def big_gemm_case(M, N, K, big, seed, a8=False, rows=None):
    rng = workloads.rng_for(seed)
    base = 4
    hi = 256 if a8 else 16
    rows = np.array([0, 1, 2, 3, M // 2, M - 1]) if rows is None else rows
    xa = rng.uniform(0.003 if a8 else 0.05, 0.2 if a8 else 3.0, M).astype(np.float32)
    xb = rng.uniform(-20.0, 0.0, M).astype(np.float32)
    codes = lambda q: dev(q.astype(np.uint8) if a8 else oq.pack_nibbles(q))
    if big == "a":  # activation row m = base row m % 4
        qa_b = rng.integers(0, hi, size=(base, K), dtype=np.int64)
        qw = rng.integers(-7, 8, size=(N, K), dtype=np.int64)
        wa = (rng.uniform(1e-3, 2e-2, N) / np.sqrt(K / 4096)).astype(np.float32)
        qa_d = codes(qa_b).repeat((M + base - 1) // base, 1)[:M]
        qw_d = dev(oq.pack_nibbles(qw))
        qa_r, qw_o, wa_o, cols = qa_b[rows % base], qw, wa, np.arange(N)
    else:  # weight row n = base row n % 4 (codes, scale and row sum)
        qa_r = rng.integers(0, hi, size=(len(rows), K), dtype=np.int64)
        qa = np.zeros((M, K), dtype=np.int8 if not a8 else np.uint8)
        qa[rows] = qa_r
        qw_o = rng.integers(-7, 8, size=(base, K), dtype=np.int64)
        wa_o = (rng.uniform(1e-3, 2e-2, base) / np.sqrt(K / 4096)).astype(np.float32)
        wa = wa_o[np.arange(N) % base]
        qa_d = codes(qa)
        del qa
        qw_d = dev(oq.pack_nibbles(qw_o)).repeat((N + base - 1) // base, 1)[:N]
        cols = np.arange(N) % base
    assert qa_d.is_contiguous() and qw_d.is_contiguous()
    assert max(qa_d.numel(), qw_d.numel()) >= 1 << 31
    rs_o = qw_o.sum(1).astype(np.int32)
    rs = rs_o[cols] if big != "a" else rs_o
    fn = sq.w4a8_linear if a8 else sq.w4a4_linear
    args = (qa_d, dev(xa), dev(xb), qw_d, dev(wa), dev(rs), None)
    y, acc = fn(*args, dbg=True)
    y2, _ = fn(*args)
    gy, gacc, gy2 = host(y), host(acc), host(y2)
    oy, oacc = olin.w4a4_linear(qa_r, xa[rows], xb[rows], qw_o, wa_o, rs_o)
    np.testing.assert_array_equal(gacc[rows], oacc[:, cols])
    parity.assert_out_close(gy[rows], oy[:, cols])
    np.testing.assert_array_equal(gy2, gy)
    del qa_d, qw_d, args
    torch.cuda.empty_cache()


@pytest.mark.slow
@pytest.mark.parametrize("M,N,K,big", [(4100, 64, (1 << 20) - 64, "a"),    # 256 x 256 register-staged tiles
                                       (100, 4100, (1 << 20) - 64, "w"),   # 128 x 128 (M <= 128)
                                       (8, 4100, (1 << 20) - 64, "w")])    # decode-sized M
def test_gemm_beyond_31bit_offsets(M, N, K, big):
    say(f"w4a4_linear M={M} N={N} K={K}: {big} operand >= 2 GB, register-staged kernel")
    big_gemm_case(M, N, K, big, seed=M + N)


@pytest.mark.slow
@pytest.mark.parametrize("M,N,K", [(16400, 64, (1 << 17) - 64),   # 128 x 64-deep tiles (K % 128 == 64)
                                   (16400, 64, 1 << 17),          # 128 x 128
                                   (16400, 1024, 1 << 17)])       # 256 x 128 (>= 512 wide tiles)
def test_w4a8_beyond_31bit_offsets(M, N, K):
    say(f"w4a8_linear M={M} N={N} K={K}: 8-bit codes >= 2 GB, register-staged kernel")
    big_gemm_case(M, N, K, "a", seed=M + N + 1, a8=True)


def tile_rows(M, tile=256):
    """Two rows of every `tile`-row block of M (its first and one inside), plus the last."""
    r = [t + o for t in range(0, M, tile) for o in (0, (37 * (t // tile + 1)) % tile) if t + o < M]
    return np.unique(np.array(r + [M - 1]))


def test_gemm_llama2_7b_down_full():
    # the launch the bench times: [2048 x 11008] x [4096 x 11008], every output column of
    # sampled rows in every M tile
    say("w4a4_linear LLaMA-2-7B down [2048x11008]x[4096x11008], rows of every M tile")
    gemm_case(2048, 4096, 11008, seed=23, bias=False, sample_rows=tile_rows(2048))


def test_gemm_llama2_7b_gate_up_stacked_full():
    say("w4a4_linear LLaMA-2-7B gate+up stacked [2048x4096]x[22016x4096], rows of every M tile")
    gemm_case(2048, 22016, 4096, seed=24, bias=False, sample_rows=tile_rows(2048))


def test_swiglu_llama2_7b_full_tiles():
    # the gate/up launch of the bench's layer step, rows in every M tile
    say("w4a4_linear_swiglu LLaMA-2-7B [2048x4096]x[2x11008x4096], rows of every M tile")
    swiglu_case(2048, 11008, 4096, seed=44, bias=False, sample_rows=tile_rows(2048))


@pytest.mark.parametrize("M,N,K", [(1, 8192, 28672), (4, 8192, 28672), (8, 4096, 11008), (16, 8192, 28672),
                                   (5, 16 * 256 * 16 - 16 * 7, 576), (100, 1000, 2112),
                                   (2048, 4096, 11008), (4096, 4096, 192)])
def test_gemm_deterministic(M, N, K):
    # dot-product decode kernel (lane sums added by DPP), LDS-streaming decode kernel (the
    # waves' partial sums of a block added in LDS), two K groups (partial sums exchanged in
    # LDS), 128 x 256 and 256 x 256 ring tiles: two launches give the same bytes
    say(f"w4a4_linear determinism M={M} N={N} K={K}")
    rng = workloads.rng_for(M + N + K + 3)
    qa = rng.integers(0, 16, size=(M, K))
    qw = rng.integers(-7, 8, size=(N, K))
    args = (dev(oq.pack_nibbles(qa)), dev(rng.uniform(0.05, 3.0, M).astype(np.float32)),
            dev(rng.uniform(-20.0, 0.0, M).astype(np.float32)), dev(oq.pack_nibbles(qw)),
            dev(rng.uniform(1e-3, 2e-2, N).astype(np.float32)), dev(qw.sum(1).astype(np.int32)))
    r = [host(sq.w4a4_linear(*args)[0]).view(np.uint16) for _ in range(2)]
    np.testing.assert_array_equal(r[0], r[1])
    a = [host(sq.w4a4_linear(*args, dbg=True)[1]) for _ in range(2)]
    np.testing.assert_array_equal(a[0], a[1])


def test_kv_and_attention_deterministic():
    say("qk_had_kvquant and attn_decode_kv4 determinism [2,512,32,128]")
    q, k, v = (dev(t) for t in workloads.kv_inputs(B=2, S=512, H=32, D=128))
    outs = [sq.qk_had_kvquant(q, k, v) for _ in range(2)]
    for name in (n for n in outs[0] if outs[0][n] is not None):
        np.testing.assert_array_equal(host(outs[0][name]).view(np.uint8), host(outs[1][name]).view(np.uint8),
                                      err_msg=name)
    o = outs[0]
    qr = o["q_rot"][:, -1].contiguous()
    cache = (o["k_q"], o["k_alpha"], o["k_beta"], o["v_q"], o["v_alpha"], o["v_beta"])
    for fn in (sq.attn_decode_kv4, sq.attn_decode_kv4_split):
        att = [host(fn(qr, *cache)).view(np.uint16) for _ in range(2)]
        np.testing.assert_array_equal(att[0], att[1])


def test_time_next_call_events():
    say("sq_time_next_call around w4a4_linear [512x1024]x[768x1024] and a rotated act quant")
    rng = workloads.rng_for(77)
    M, N, K = 512, 768, 1024
    qa = rng.integers(0, 16, size=(M, K))
    qw = rng.integers(-7, 8, size=(N, K))
    args = (dev(oq.pack_nibbles(qa)), dev(rng.uniform(0.1, 1, M).astype(np.float32)),
            dev(rng.uniform(-5, 0, M).astype(np.float32)), dev(oq.pack_nibbles(qw)),
            dev(rng.uniform(1e-3, 1e-2, N).astype(np.float32)), dev(qw.sum(1).astype(np.int32)))
    ref, _ = sq.w4a4_linear(*args)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    sq.time_next_call(a, b)
    y, _ = sq.w4a4_linear(*args)
    y2, _ = sq.w4a4_linear(*args)  # not timed: the events were consumed
    torch.cuda.synchronize()
    ms = a.elapsed_time(b)
    assert 0 < ms < 50
    assert torch.equal(y, ref) and torch.equal(y2, ref)
    x = dev(workloads.outlier_acts(rng, 64, 28 * 512, 8, 50.0))
    q0 = sq.had_quant_act(x, had_table(28), 512)[0]
    sq.time_next_call(a, b)
    q1 = sq.had_quant_act(x, had_table(28), 512)[0]
    torch.cuda.synchronize()
    assert 0 < a.elapsed_time(b) < 50
    assert torch.equal(q0, q1)
