"""The allocation-free decode attention (sq_attn_decode_kv4_split_noalloc) against the
workspace entry point (sq_attn_decode_kv4_split) it shares its kernels with: equal bytes,
on two calls in a row through the C ABI, the second on a smaller cache."""

import ctypes

import numpy as np
import pytest
import torch

from oracle import kv as okv
from oracle import quant as oq
from paper_2405_16406_amd import sq, workloads

import parity

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def cache(B, S, H, seed):
    rng = workloads.rng_for(seed)
    kc, vc = rng.integers(0, 16, (B, S, H, 128)), rng.integers(0, 16, (B, S, H, 128))
    ka, va = (rng.uniform(0.01, 0.2, (B, S, H)).astype(np.float32) for _ in range(2))
    kb, vb = (rng.uniform(-1.5, 0.0, (B, S, H)).astype(np.float32) for _ in range(2))
    q = (rng.standard_normal((B, H, 128)) * 2).astype(np.float16)
    return [q, oq.pack_nibbles(kc), ka, kb, oq.pack_nibbles(vc), va, vb]


def noalloc(args, out):
    L = sq.lib()
    q, kq, ka, kb, vq, va, vb = args
    B, H, D = q.shape
    st = L.sq_attn_decode_kv4_split_noalloc(*(ctypes.c_void_p(t.data_ptr()) for t in args), B, kq.shape[1], H, D,
                                            ctypes.c_float(1.0 / D ** 0.5), 32, ctypes.c_void_p(out.data_ptr()),
                                            ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == sq.SQ_OK, sq.lib().sq_last_error()


def test_noalloc_matches_workspace_entry_point():
    for (B, S, H), seed in (((8, 2048, 32), 900), ((2, 700, 5), 901)):
        print(f"[gpu case] attn_decode_kv4_split_noalloc B={B} S={S} H={H}", flush=True)
        host_args = cache(B, S, H, seed)
        args = [torch.from_numpy(np.ascontiguousarray(a)).to(DEV) for a in host_args]
        out = torch.empty_like(args[0])
        noalloc(args, out)
        ref = sq.attn_decode_kv4_split(*args)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        np.testing.assert_array_equal(got.view(np.uint16), ref.cpu().numpy().view(np.uint16))
        if B * S * H <= 10000:
            parity.assert_out_close(got, okv.attn_decode(*host_args))
