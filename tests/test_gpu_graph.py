"""The hot path inside a HIP graph: the library's launches take the caller's stream and
allocate nothing, so a decode step (activation quant -> gate/up with SiLU -> R4 + quant ->
down) and the allocation-free split decode attention can be captured once and replayed.
Every replay is checked bit for bit against the eager calls, with eager work and
synchronisations between the replays and new inputs copied into the captured buffers."""

import numpy as np
import pytest
import torch

from paper_2405_16406_amd import sq, workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def up(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


@pytest.mark.parametrize("M", [1, 4])
def test_decode_step_graph_replays_match_eager(M):
    # M = 1: the dot-product decode kernels; M = 4: the 16-row decode kernels
    shape = workloads.LLAMA2_7B_MLP
    H, I = shape.hidden, shape.inter
    print(f"[gpu case] graph of a decode step M={M}, LLaMA-2-7B MLP", flush=True)
    inp = workloads.mlp_inputs(shape, rows=3 * M)
    had = up(sq.hadamard_factor(shape.had_dense))
    wsw = sq.pack_w4(sq.interleave_gate_up(up(inp["w_gate"]), up(inp["w_up"])).contiguous())
    wd = sq.pack_w4(up(inp["w_down"]), had, shape.had_pow2)
    xs = [up(inp["x_in"][k * M:(k + 1) * M]) for k in range(3)]
    x = xs[0].clone()  # the captured input buffer
    xq = (torch.empty((M, H // 2), dtype=torch.uint8, device=DEV),
          torch.empty((M, 1), dtype=torch.float32, device=DEV), torch.empty((M, 1), dtype=torch.float32, device=DEV))
    hq = (torch.empty((M, I // 2), dtype=torch.uint8, device=DEV),
          torch.empty((M, 1), dtype=torch.float32, device=DEV), torch.empty((M, 1), dtype=torch.float32, device=DEV))
    h = torch.empty((M, I), dtype=torch.float16, device=DEV)
    y = torch.empty((M, H), dtype=torch.float16, device=DEV)

    def step():
        sq.had_quant_act(x, out=xq)
        sq.w4a4_linear_swiglu(*xq, *wsw, out=h)
        sq.had_quant_act(h, had, shape.had_pow2, out=hq)
        sq.w4a4_linear(*hq, *wd, out=y)

    def eager(xin):
        x.copy_(xin)
        step()
        torch.cuda.synchronize()
        return y.clone()

    refs = [eager(t) for t in xs]
    assert not torch.equal(refs[0], refs[1])
    g = torch.cuda.CUDAGraph()
    x.copy_(xs[0])
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        k = rep % 3
        x.copy_(xs[k])
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.cpu().numpy().view(np.uint16), refs[k].cpu().numpy().view(np.uint16),
                                      err_msg=f"replay {rep}")
        # eager work between the replays, on other data
        other = eager(xs[(k + 1) % 3])
        np.testing.assert_array_equal(other.cpu().numpy().view(np.uint16),
                                      refs[(k + 1) % 3].cpu().numpy().view(np.uint16))


def test_noalloc_attention_graph_replays_match_eager():
    B, S, H = 2, 1000, 32
    print(f"[gpu case] graph of attn_decode_kv4_split_noalloc B={B} S={S} H={H}", flush=True)
    q, k, v = (up(t) for t in workloads.kv_inputs(B=B, S=S, H=H, D=128))
    o = sq.qk_had_kvquant(q, k, v)
    cache = [o[n] for n in ("k_q", "k_alpha", "k_beta", "v_q", "v_alpha", "v_beta")]
    qs = [o["q_rot"][:, t].contiguous() for t in (S - 1, S - 2, S - 3)]
    qr = qs[0].clone()
    out = torch.empty_like(qr)
    refs = [sq.attn_decode_kv4_split(t, *cache).clone() for t in qs]
    sq.attn_decode_kv4_split_noalloc(qr, *cache, out=out)  # first call: the scratch's address
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sq.attn_decode_kv4_split_noalloc(qr, *cache, out=out)
    for rep in range(4):
        j = rep % 3
        qr.copy_(qs[j])
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(out.cpu().numpy().view(np.uint16), refs[j].cpu().numpy().view(np.uint16),
                                      err_msg=f"replay {rep}")
        e = sq.attn_decode_kv4_split_noalloc(qs[(j + 1) % 3], *cache)  # eager, same scratch
        torch.cuda.synchronize()
        np.testing.assert_array_equal(e.cpu().numpy().view(np.uint16), refs[(j + 1) % 3].cpu().numpy().view(np.uint16))
