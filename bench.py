"""Benchmark of the rotated W4A4 hot path on one MI355X.

One step = one pass of the whole path over one LLaMA-2-7B transformer layer's worth of
tokens (M = 2048), chained as the layer runs it:
  1. R3 + 4-bit KV quantization of Q, K, V [1, 2048, 32, 128]          sq_qk_had_kvquant
  2. per-token 4-bit quantization of the MLP input x [2048, 4096]        sq_had_quant_act (identity)
  3. gate and up projections in one product, SiLU(g) * u in the
     epilogue: h [2048, 11008] = [2048x4096] x [2x11008x4096]^T           sq_w4a4_linear_swiglu
  4. online R4 (H_172 (x) S_64) + 4-bit quantization of h                 sq_had_quant_act
  5. down projection [2048x11008] x [4096x11008]^T                       sq_w4a4_linear
Weights are packed once beforehand (sq_pack_w4; R4 folded into W_down; gate and up rows
interleaved in blocks of 32), as in deployment.  Inputs are synthetic (seeded,
LLaMA-shaped, with outlier channels) and already resident in HBM; eight input/weight sets
(--sets) are rotated so that consecutive steps do not find the previous step's weights in
the 256 MB Infinity Cache.

value = W4A4 linear ops of the step (3 x 2*M*N*K) / step time, in TOPS.  Per-kernel
durations come from a second pass over the same steps, in which the library attaches a
pair of HIP events to its own kernel launches (start/stop of the launch, on the stream it
runs on).  `roofline` is for the dominant kernel (the gate/up product).

`configs` times every kernel of every workload on its own (LLaMA-2-7B, LLaMA-3-8B, the
R3 + KV cache [8, 2048, 32, 128] and its decode attention, LLaMA-2-70B decode at M = 1, 8,
16, the tiny case), each launch on its own copies of its operands so that nothing is
served from a cache, with its algorithmic bytes or ops and its roofline fraction.
`peaks` are what this machine sustains: an int8 matrix-core loop, a copy and a read stream.
The CPU baseline times the oracle on a bounded slice of the step.

    python bench.py [--steps K] [--warmup W] [--no-cpu] [--no-configs] [--only NAME]
"""

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "W4A4 rotated-linear TOPS + Hadamard/quant GB/s at LLaMA-2-7B/3-8B shapes"
HBM_PEAK_GBS = 8000.0    # MI355X HBM3E
INT8_PEAK_TOPS = 5000.0  # MI355X dense int8 matrix cores
CSRC = os.path.join(ROOT, "paper_2405_16406_amd", "csrc")
PROFILE_DIR = os.path.join(ROOT, "profiles")
TRAFFIC_FILE = os.path.join(PROFILE_DIR, "hbm_traffic.json")
SPAN_BYTES = 1 << 30    # bytes each isolated kernel cycles through (4x the Infinity Cache)
CALIB_BYTES = 512 << 20  # bytes read and written by each --calib-copy launch
ONLY = ("step", "peaks", "c1", "c2", "c3", "c4", "c5", "variants")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=30)
    p.add_argument("--sets", type=int, default=8, help="input/weight sets rotated between steps")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU oracle time")
    p.add_argument("--no-configs", action="store_true", help="skip the per-config kernel timings and peaks")
    p.add_argument("--only", choices=ONLY, default=None,
                   help="run one part (for profiling runs); prints its results")
    p.add_argument("--calib-copy", action="store_true",
                   help="only run a plain 512 MiB copy kernel four times (counter calibration) and exit")
    p.add_argument("--summarize", default=None, metavar="DIR",
                   help="write the profiles/ summaries from rocprofv3 outputs under DIR and exit (no GPU)")
    return p.parse_args()


# ---------------------------------------------------------------- algorithmic work

def gemm_bytes(M, N, K, out_cols=None):
    """Packed operands, fp16 output [M, out_cols] (N unless the epilogue halves it), scales."""
    out_cols = N if out_cols is None else out_cols
    return M * K // 2 + N * K // 2 + 2 * M * out_cols + 8 * (M + N)


def gemm8_bytes(M, N, K):
    return M * K + N * K // 2 + 2 * M * N + 8 * (M + N)


def had_bytes(M, K, bits=4, groups_per_row=1):
    return 2 * M * K + M * K * bits // 8 + 8 * M * groups_per_row


def kv_bytes(E, bits=4, param_bytes=4):
    """Q, K, V in (fp16); Q_rot out (fp16); K, V codes; four group parameters per 128."""
    return 3 * 2 * E + 2 * E + 2 * (E * bits // 8) + 4 * param_bytes * (E // 128)


def attn_bytes(B, S, H, D=128, param_bytes=4):
    """Decode attention over a 4-bit cache: K and V codes and their four group parameters
    per cached (token, head), plus the fp16 query and output per head."""
    return B * S * H * (2 * (D // 2) + 4 * param_bytes) + 2 * B * H * D * 2


def entry(ms, work, kind, bound=None):
    """One kernel's record: kind 'ops' (MFMA-bound, TOP/s vs int8 peak) or 'bytes' (HBM)."""
    t = ms * 1e-3
    if kind == "ops":
        ach = work / t / 1e12
        return {"us": round(ms * 1e3, 2), "ops": int(work), "achieved": round(ach, 1), "unit": "TOP/s",
                "bound": bound or "mfma", "peak": INT8_PEAK_TOPS, "frac": round(ach / INT8_PEAK_TOPS, 4)}
    ach = work / t / 1e9
    return {"us": round(ms * 1e3, 2), "bytes": int(work), "achieved": round(ach, 1), "unit": "GB/s",
            "bound": bound or "hbm", "peak": HBM_PEAK_GBS, "frac": round(ach / HBM_PEAK_GBS, 4)}


# ---------------------------------------------------------------- measured HBM traffic

def source_hash(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


# bench kernel -> (profiled part, kernel name as the summaries shorten it, grid in threads)
# of its launches in the rocprofv3 runs of PROFILE_COMMANDS; filled from those runs' kernel
# tables.  A kernel reports measured traffic only while the source the counters were taken
# on is unchanged (hbm_traffic.json keeps its hash).
TRAFFIC_MAP = {
    "c2/kv_quant": ("step", "qk_had_kvquant_v2<false, 4, false>", 262144),
    "c2/act_quant": ("step", "quant_rows_identity<4, 2>", 524288),
    "c2/gate_up_swiglu": ("step", "w4a4_gemm_ring<2, 4, 4, 2, 4, 1, 1, false>", 352256),
    "c2/r4_had_quant": ("step", "had_quant_pair<172, 176, 6, false, 4, false>", 131072),
    "c2/down_gemm": ("step", "w4a4_gemm_ring<2, 4, 2, 2, 3, 1, 1, false>", 131072),
    "c3/act_quant": ("c3", "quant_rows_identity<4, 2>", 1048576),
    "c3/gate_up_swiglu": ("c3", "w4a4_gemm_ring<2, 4, 4, 2, 4, 1, 1, false>", 917504),
    "c3/r4_had_quant": ("c3", "had_quant_lines<28, 8, 7, false, 4, false>", 229376),
    "c3/down_gemm": ("c3", "w4a4_gemm_ring<2, 4, 4, 2, 4, 1, 1, false>", 131072),
    "c4/kv_quant": ("c4", "qk_had_kvquant_v2<true, 4, false>", 2097152),
    "c4/attn_decode": ("c4", "attn_decode_kv4<false>", 262144),
    # two kernels (on 256 CUs: 16 chunks x 2 groups of 16 heads x 8 batches of 8 waves,
    # then one workgroup of one wave per head)
    "c4/attn_decode_split": [("c4", "attn_decode_part<false, false, 8, 1, 2, 2>", 131072),
                             ("c4", "attn_decode_combine", 16384)],
}
for _m, _g in ((1, 256), (8, 2048), (16, 4096)):  # the decode sizes share the GEMM launch shapes
    TRAFFIC_MAP[f"c5m{_m}/act_quant"] = ("c5", "quant_rows_identity<4, 4>", _g)
    TRAFFIC_MAP[f"c5m{_m}/r4_had_quant"] = ("c5", "had_quant_lines<28, 16, 14, false, 4, false>", 896 * _m)
    # M = 1: the dot-product kernel, 8 waves on each of the 256 CUs; M = 8 and 16: the
    # LDS-streaming kernel (gate/up: 256 workgroups of 7 gate/up block pairs; down: 256 of 2
    # blocks)
    TRAFFIC_MAP[f"c5m{_m}/gate_up_swiglu"] = (("c5", "w4a4_gemv<1, true, false>", 131072) if _m == 1 else
                                              ("c5", "w4a4_gemm_stream<256, 2, true, false>", 131072))
    TRAFFIC_MAP[f"c5m{_m}/down_gemm"] = (("c5", "w4a4_gemv<1, false, false>", 131072) if _m == 1 else
                                         ("c5", "w4a4_gemm_stream<256, 2, false, false>", 131072))


def measured_traffic(key):
    """HBM bytes per launch of bench kernel `key` (e.g. 'c2/gate_up_swiglu') from the
    committed rocprofv3 FETCH_SIZE/WRITE_SIZE runs, if they were taken on the current source."""
    if key not in TRAFFIC_MAP:
        return None
    launches = TRAFFIC_MAP[key] if isinstance(TRAFFIC_MAP[key], list) else [TRAFFIC_MAP[key]]
    try:
        with open(TRAFFIC_FILE) as f:
            by_grid = json.load(f)["by_grid"]
    except (OSError, ValueError, KeyError):
        return None
    rd = wr = 0
    for launch in launches:  # a call of several kernels: their bytes add up
        t = by_grid.get("|".join(str(v) for v in launch))
        if not t or t.get("source_sha256_16") != source_hash(os.path.join(CSRC, t["source"])):
            return None
        rd, wr = rd + t["read_bytes"], wr + t["write_bytes"]
    return {"read": rd, "write": wr, "total": rd + wr}


# ---------------------------------------------------------------- roofline probes

class Probe:
    """libsq_probe.so (include/sq_probe.h)."""

    def __init__(self):
        path = os.path.join(ROOT, "paper_2405_16406_amd", "libsq_probe.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with `python -m paper_2405_16406_amd.build`")
        L = ctypes.CDLL(path)
        P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        L.sq_probe_last_error.restype = ctypes.c_char_p
        L.sq_probe_mfma_i8.restype = I32
        L.sq_probe_mfma_i8.argtypes = [I64, I32, I32, P, P]
        L.sq_probe_copy.restype = I32
        L.sq_probe_copy.argtypes = [P, P, I64, I32, P]
        L.sq_probe_read.restype = I32
        L.sq_probe_read.argtypes = [P, I64, I32, P, P]
        L.sq_probe_copy_blocks.restype = I32
        L.sq_probe_copy_blocks.argtypes = [P, P, I64, I32, P]
        L.sq_probe_read_blocks.restype = I32
        L.sq_probe_read_blocks.argtypes = [P, I64, I32, P, P]
        L.sq_probe_sleep.restype = I32
        L.sq_probe_sleep.argtypes = [I64, P]
        self.L = L

    def check(self, status, what):
        if status != 0:
            raise RuntimeError(f"{what}: {self.L.sq_probe_last_error().decode()}")

    def hold(self, torch, ms):
        """Hold the current stream for about `ms` milliseconds (one sleeping wave), so that
        the launches the host queues next run back to back."""
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        self.check(self.L.sq_probe_sleep(int(ms * 1000), stream), "sleep probe")


_PROBE = None


def probe():
    global _PROBE
    if _PROBE is None:
        _PROBE = Probe()
    return _PROBE


def measure_peaks(torch, dev):
    """What this machine sustains: int8 MFMA loop (TOP/s), copy and read streams (GB/s)."""
    pr = probe()
    stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ts = []
        for _ in range(reps):
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    out = {}
    iters = 4096
    for wps in (1, 2):
        wg = 256  # one workgroup per CU: wps waves on each SIMD
        sink = torch.empty(wg * 256 * wps, dtype=torch.int32, device=dev)
        ms = timed(lambda: pr.check(pr.L.sq_probe_mfma_i8(iters, wg, wps, ctypes.c_void_p(sink.data_ptr()), stream),
                                    "mfma probe"), 5)
        ops = 65536 * 8 * iters * wg * 4 * wps
        out[f"mfma_i8_{wps}_waves_per_simd"] = {"TOPs": round(ops / (ms * 1e-3) / 1e12, 1), "us": round(ms * 1e3, 1)}
    nbytes = 1 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(3)
    dst = torch.empty_like(src)
    sink = torch.empty(2048 * 256, dtype=torch.int32, device=dev)
    sp, dp = ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr())
    for wg in (1024, 2048, 8192):
        sk = torch.empty(wg * 256, dtype=torch.int32, device=dev)
        skp = ctypes.c_void_p(sk.data_ptr())
        for kind, fn in (("", pr.L.sq_probe_copy), ("blocks_", pr.L.sq_probe_copy_blocks)):
            ms = timed(lambda: pr.check(fn(sp, dp, nbytes, wg, stream), "copy probe"), 5)
            out[f"copy_{kind}{wg}_workgroups"] = {"GBps": round(2 * nbytes / (ms * 1e-3) / 1e9, 1),
                                                  "us": round(ms * 1e3, 1)}
        for kind, fn in (("", pr.L.sq_probe_read), ("blocks_", pr.L.sq_probe_read_blocks)):
            ms = timed(lambda: pr.check(fn(sp, nbytes, wg, skp, stream), "read probe"), 5)
            out[f"read_{kind}{wg}_workgroups"] = {"GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
                                                  "us": round(ms * 1e3, 1)}
    del src, dst, sink
    torch.cuda.empty_cache()
    # the ROCm library's int8 GEMM (torch._int_mm -> hipBLASLt) on int8 operands of the MLP
    # shapes, codes in [-8, 8): what a vendor kernel sustains on the same matrix cores
    # (twice the operand bytes of the packed 4-bit kernels, no nibble expansion)
    vendor = {}
    for (M, N, K) in ((2048, 22016, 4096), (2048, 4096, 11008), (4096, 28672, 4096), (4096, 4096, 14336)):
        try:
            g = torch.Generator(device=dev).manual_seed(M + N + K)
            a = torch.randint(-8, 8, (M, K), dtype=torch.int8, device=dev, generator=g)
            bt = torch.randint(-8, 8, (N, K), dtype=torch.int8, device=dev, generator=g).t()
            ms = timed(lambda: torch._int_mm(a, bt), 10)
            vendor[f"{M}x{N}x{K}"] = {"TOPs": round(2 * M * N * K / (ms * 1e-3) / 1e12, 1), "us": round(ms * 1e3, 1)}
            del a, bt
        except (RuntimeError, AttributeError) as e:  # an operator missing from this torch build
            vendor[f"{M}x{N}x{K}"] = {"error": str(e)[:120]}
    torch.cuda.empty_cache()
    best = lambda pre, f: max(v[f] for k, v in out.items() if k.startswith(pre))
    return {"int8_mfma_TOPs": best("mfma", "TOPs"), "copy_GBps": best("copy", "GBps"), "read_GBps": best("read", "GBps"),
            "datasheet": {"int8_mfma_TOPs": INT8_PEAK_TOPS, "hbm_GBps": HBM_PEAK_GBS},
            "runs": out,
            "vendor_int8_gemm": vendor,
            "note": "int8 loop: back-to-back v_mfma_i32_32x32x32_i8 on registers with int4-code operand bytes, "
                    "8 accumulators per wave; copy GB/s counts bytes read + written; copy/read: grid-stride 16-byte "
                    "accesses, blocks_: each workgroup streams its own contiguous region; median of 5 launches"}


# ---------------------------------------------------------------- the chained layer step

def run_step(args, torch, sq, workloads, dev):
    shape = workloads.LLAMA2_7B_MLP
    M, HID, INTER = shape.M, shape.hidden, shape.inter
    A, B = shape.had_dense, shape.had_pow2
    NH, HD = 32, 128
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    had = up(sq.hadamard_factor(A))

    # resident inputs: `sets` distinct sets of activations and packed weights.  Set 0 comes
    # from the seeded generators; set s > 0 is set 0 with its rows rotated by s * 997
    # (tokens for activations, output channels for weights): same distributions.
    inp = workloads.mlp_inputs(shape, rows=M)
    rng = workloads.rng_for(500)
    base = dict(x_in=up(inp["x_in"]), qkv=[up(workloads.head_acts(rng, 1, M, NH, HD, 2, 30.0)) for _ in range(3)],
                w_g=up(inp["w_gate"]), w_u=up(inp["w_up"]), w_down=up(inp["w_down"]))
    del inp
    sets = []
    for s in range(args.sets):
        r = lambda t, dim=0: torch.roll(t, shifts=s * 997, dims=dim).contiguous()
        wsw = sq.interleave_gate_up(r(base["w_g"]), r(base["w_u"])).contiguous()
        sets.append(dict(x_in=r(base["x_in"]), qkv=[r(t, 1) for t in base["qkv"]],
                         wsw=sq.pack_w4(wsw), wd=sq.pack_w4(r(base["w_down"]), had, B)))
        del wsw
    del base
    torch.cuda.synchronize()

    kv_out = dict(q_rot=torch.empty((1, M, NH, HD), dtype=torch.float16, device=dev),
                  k_q=torch.empty((1, M, NH, HD // 2), dtype=torch.uint8, device=dev),
                  k_alpha=torch.empty((1, M, NH, 1), dtype=torch.float32, device=dev),
                  k_beta=torch.empty((1, M, NH, 1), dtype=torch.float32, device=dev),
                  v_q=torch.empty((1, M, NH, HD // 2), dtype=torch.uint8, device=dev),
                  v_alpha=torch.empty((1, M, NH, 1), dtype=torch.float32, device=dev),
                  v_beta=torch.empty((1, M, NH, 1), dtype=torch.float32, device=dev))
    codes = lambda K: (torch.empty((M, K // 2), dtype=torch.uint8, device=dev),
                       torch.empty((M, 1), dtype=torch.float32, device=dev),
                       torch.empty((M, 1), dtype=torch.float32, device=dev))
    xq_in, xq_dn = codes(HID), codes(INTER)
    h = torch.empty((M, INTER), dtype=torch.float16, device=dev)
    y_dn = torch.empty((M, HID), dtype=torch.float16, device=dev)

    names = ["kv_quant", "act_quant", "gate_up_swiglu", "r4_had_quant", "down_gemm"]

    def calls(s):
        d = sets[s]
        return [
            lambda: sq.qk_had_kvquant(*d["qkv"], out=kv_out),
            lambda: sq.had_quant_act(d["x_in"], out=xq_in),
            lambda: sq.w4a4_linear_swiglu(*xq_in, *d["wsw"], out=h),
            lambda: sq.had_quant_act(h, had, B, out=xq_dn),
            lambda: sq.w4a4_linear(*xq_dn, *d["wd"], out=y_dn),
        ]

    step_calls = [calls(s) for s in range(args.sets)]

    def step(s):
        for c in step_calls[s]:
            c()

    for w in range(args.warmup):
        step(w % args.sets)
    torch.cuda.synchronize()

    # timed region: K whole steps back to back, nothing recorded between kernels
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record()
    for k in range(args.steps):
        step(k % args.sets)
    t_end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t_start.elapsed_time(t_end) / args.steps

    # per-kernel durations inside the step: the same K steps again, each call timed by a
    # pair of HIP events the library attaches to its own kernel launch (sq_time_next_call);
    # kept out of the timed region: arming the events costs host time per call
    ev = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)] for _ in names]
          for _ in range(args.steps)]
    for k in range(args.steps):
        for i in range(len(names)):
            for e in ev[k][i]:
                e.record()  # creates the HIP events
    torch.cuda.synchronize()
    for k in range(args.steps):
        for i, c in enumerate(step_calls[k % args.sets]):
            sq.time_next_call(ev[k][i][0], ev[k][i][1])
            c()
    torch.cuda.synchronize()
    per = {n: float(np.mean([ev[k][i][0].elapsed_time(ev[k][i][1]) for k in range(args.steps)]))
           for i, n in enumerate(names)}

    gemm_ops = 2 * M * INTER * HID
    E = M * NH * HD
    kernels = {
        "kv_quant": entry(per["kv_quant"], kv_bytes(E), "bytes"),
        "act_quant": entry(per["act_quant"], had_bytes(M, HID), "bytes"),
        "gate_up_swiglu": entry(per["gate_up_swiglu"], 2 * gemm_ops, "ops"),
        "r4_had_quant": entry(per["r4_had_quant"], had_bytes(M, INTER), "bytes"),
        "down_gemm": entry(per["down_gemm"], gemm_ops, "ops"),
    }
    kernels["gate_up_swiglu"]["algorithmic_bytes"] = gemm_bytes(M, 2 * INTER, HID, out_cols=INTER)
    kernels["down_gemm"]["algorithmic_bytes"] = gemm_bytes(M, HID, INTER)
    for n, k_ in kernels.items():
        k_["traffic"] = measured_traffic(f"c2/{n}")
    del sets, step_calls
    torch.cuda.empty_cache()
    return dict(ms_step=ms_step, wall=wall, per=per, kernels=kernels, step_ops=3 * gemm_ops,
                shape=shape, names=names)


# ---------------------------------------------------------------- isolated kernels per config

def n_copies(nbytes):
    return int(min(32, max(2, -(-SPAN_BYTES // max(nbytes, 1)))))


def timed_calls(torch, sq, fns, reps=None):
    """Mean kernel time per launch over back-to-back launches cycling through fns, each
    timed by the call's own start/end events (sq_time_next_call).  A sleeping wave holds
    the stream while the host queues the launches, so they run back to back on the GPU
    (a host-paced launch would time an idle GPU's start-up)."""
    reps = reps or max(20, 2 * len(fns))
    for f in fns:
        f()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in evs:
        a.record()
        b.record()
    torch.cuda.synchronize()
    probe().hold(torch, 2.0 + 0.3 * reps)
    for r in range(reps):
        sq.time_next_call(*evs[r])
        fns[r % len(fns)]()
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in evs) / reps


class Cfg:
    """Timing helpers over distinct copies of each kernel's operands (> 1 GB in all)."""

    def __init__(self, torch, sq, dev):
        self.torch, self.sq, self.dev = torch, sq, dev

    def act(self, x, had, pow2, nbytes, bits=4, **var):
        sq = self.sq
        fns = []
        for _ in range(n_copies(nbytes)):
            xc = x.clone()
            o = sq.had_quant_act(xc, had, pow2, bits=bits, **var)[:3]
            fns.append(lambda xc=xc, o=o: sq.had_quant_act(xc, had, pow2, bits=bits, out=o, **var))
        return timed_calls(self.torch, sq, fns)

    def gemm(self, qx, w, nbytes, kind="w4a4"):
        sq = self.sq
        fns = []
        for _ in range(n_copies(nbytes)):
            qc = tuple(t.clone() for t in qx)
            wc = tuple(t.clone() for t in w)
            if kind == "swiglu":
                y = sq.w4a4_linear_swiglu(*qc, *wc)
                fns.append(lambda qc=qc, wc=wc, y=y: sq.w4a4_linear_swiglu(*qc, *wc, out=y))
            elif kind == "w4a8":
                y = sq.w4a8_linear(*qc, *wc)[0]
                fns.append(lambda qc=qc, wc=wc, y=y: sq.w4a8_linear(*qc, *wc, out=y))
            else:
                y = sq.w4a4_linear(*qc, *wc)[0]
                fns.append(lambda qc=qc, wc=wc, y=y: sq.w4a4_linear(*qc, *wc, out=y))
        return timed_calls(self.torch, sq, fns)


def mlp_config(tag, shape, torch, sq, workloads, dev, variants=False, inp=None, tokens=None):
    """Isolated kernels of one MLP layer: act quant, gate/up with SiLU, R4 + quant, down."""
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    C = Cfg(torch, sq, dev)
    inp = workloads.mlp_inputs(shape) if inp is None else inp
    M = shape.M if tokens is None else tokens
    H, I = shape.hidden, shape.inter
    had = up(sq.hadamard_factor(shape.had_dense))
    xin, xdn = up(inp["x_in"][:M]), up(inp["x_down"][:M])
    wsw = sq.pack_w4(sq.interleave_gate_up(up(inp["w_gate"]), up(inp["w_up"])).contiguous())
    wd = sq.pack_w4(up(inp["w_down"]), had, shape.had_pow2)
    qi = sq.had_quant_act(xin)[:3]
    qd = sq.had_quant_act(xdn, had, shape.had_pow2)[:3]
    b_aq, b_hq = had_bytes(M, H), had_bytes(M, I)
    b_sw, b_d = gemm_bytes(M, 2 * I, H, out_cols=I), gemm_bytes(M, H, I)
    ops_sw, ops_d = 4 * M * I * H, 2 * M * I * H
    decode = M <= 16
    k = {}
    k["act_quant"] = entry(C.act(xin, None, 1, b_aq), b_aq, "bytes", "latency" if decode else "hbm")
    t = C.gemm(qi, wsw, b_sw, "swiglu")
    k["gate_up_swiglu"] = entry(t, b_sw, "bytes") if decode else entry(t, ops_sw, "ops")
    k["gate_up_swiglu"].update({"ops": ops_sw} if decode else {"algorithmic_bytes": b_sw})
    t = C.act(xdn, had, shape.had_pow2, b_hq)
    k["r4_had_quant"] = entry(t, b_hq, "bytes", "latency" if decode else "hbm")
    t = C.gemm(qd, wd, b_d)
    k["down_gemm"] = entry(t, b_d, "bytes") if decode else entry(t, ops_d, "ops")
    k["down_gemm"].update({"ops": ops_d} if decode else {"algorithmic_bytes": b_d})
    if variants:
        # W4A8 (8-bit activation codes into the same weights), and R4 with a random-sign
        # Hadamard S H and a clipped range (S: K bytes per row set from cache, not counted)
        qi8 = sq.had_quant_act(xin, bits=8)[:3]
        qd8 = sq.had_quant_act(xdn, had, shape.had_pow2, bits=8)[:3]
        wgu = sq.pack_w4(torch.cat([up(inp["w_gate"]), up(inp["w_up"])]))
        b8_hq, b8_gu, b8_d = had_bytes(M, I, 8), gemm8_bytes(M, 2 * I, H), gemm8_bytes(M, H, I)
        k["r4_had_quant_8bit"] = entry(C.act(xdn, had, shape.had_pow2, b8_hq, bits=8), b8_hq, "bytes")
        t = C.gemm(qi8, wgu, b8_gu, "w4a8")
        k["gate_up_w4a8"] = entry(t, b8_gu, "bytes") if decode else entry(t, ops_sw, "ops")
        t = C.gemm(qd8, wd, b8_d, "w4a8")
        k["down_w4a8"] = entry(t, b8_d, "bytes") if decode else entry(t, ops_d, "ops")
        sgn = up(np.where(workloads.rng_for(7).random(I) < 0.5, -1, 1).astype(np.int8))
        k["r4_had_quant_signs_clip"] = entry(C.act(xdn, had, shape.had_pow2, b_hq, signs=sgn, clip=0.9), b_hq,
                                             "bytes")
    for n, e in k.items():
        e["traffic"] = measured_traffic(f"{tag}/{n}")
    res = {"workload": shape.name if tokens is None else f"{shape.name.split(',')[0]}, M={M}", "kernels": k}
    if decode:
        res["chained_step"] = decode_chain(torch, sq, xin, had, shape.had_pow2, wsw, wd)
    torch.cuda.empty_cache()
    return res


def decode_chain(torch, sq, x, had, pow2, wsw, wd, reps=50):
    """The decode MLP step chained (act quant -> gate/up with SiLU -> R4 + quant -> down) on
    preallocated buffers: mean time per step over `reps` back-to-back steps, launched
    eagerly and as the replay of one captured HIP graph."""
    M, H = x.shape
    I = wd[0].shape[1] * 2
    dev = x.device
    xq = (torch.empty((M, H // 2), dtype=torch.uint8, device=dev), torch.empty((M, 1), dtype=torch.float32, device=dev),
          torch.empty((M, 1), dtype=torch.float32, device=dev))
    hq = (torch.empty((M, I // 2), dtype=torch.uint8, device=dev), torch.empty((M, 1), dtype=torch.float32, device=dev),
          torch.empty((M, 1), dtype=torch.float32, device=dev))
    h = torch.empty((M, I), dtype=torch.float16, device=dev)
    y = torch.empty((M, H), dtype=torch.float16, device=dev)

    def step():
        sq.had_quant_act(x, out=xq)
        sq.w4a4_linear_swiglu(*xq, *wsw, out=h)
        sq.had_quant_act(h, had, pow2, out=hq)
        sq.w4a4_linear(*hq, *wd, out=y)

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        probe().hold(torch, 2.0 + 0.05 * reps)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e3

    eager_us = timed(step)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    graph_us = timed(g.replay)
    del g
    return {"eager_us": round(eager_us, 2), "graph_us": round(graph_us, 2), "steps": reps,
            "note": "four library calls per step; weights are read from HBM each step (352 MB > the 256 MB "
                    "Infinity Cache)"}


def kv_config(torch, sq, workloads, dev, variants=False):
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    q, k, v = (up(t) for t in workloads.kv_inputs())
    E = q.numel()
    B, S, H, D = q.shape

    def kv_fns(nbytes, **kw):
        fns = []
        for _ in range(n_copies(nbytes)):
            qc, kc, vc = q.clone(), k.clone(), v.clone()
            o = sq.qk_had_kvquant(qc, kc, vc, **kw)
            o.pop("k_rot")
            fns.append(lambda qc=qc, kc=kc, vc=vc, o=o: sq.qk_had_kvquant(qc, kc, vc, out=o, **kw))
        return fns

    def attn_fns(nbytes, split=False, **kw):
        # split: sq_attn_decode_kv4_split with one workspace (the calls are ordered on the stream)
        ws = torch.empty(max(sq.attn_decode_workspace_bytes(B, S, H, D), 1), dtype=torch.uint8, device=dev)
        fns = []
        for _ in range(n_copies(nbytes)):
            o = sq.qk_had_kvquant(q, k, v, **kw)
            qr = o["q_rot"][:, -1].contiguous()
            oa = torch.empty_like(qr)
            cache = (o["k_q"], o["k_alpha"], o["k_beta"], o["v_q"], o["v_alpha"], o["v_beta"])
            if split:
                fns.append(lambda qr=qr, cache=cache, oa=oa: sq.attn_decode_kv4_split(qr, *cache, out=oa,
                                                                                       workspace=ws))
            else:
                fns.append(lambda qr=qr, cache=cache, oa=oa: sq.attn_decode_kv4(qr, *cache, out=oa))
        return fns

    kk = {}
    b = kv_bytes(E)
    kk["kv_quant"] = entry(timed_calls(torch, sq, kv_fns(b)), b, "bytes")
    b = attn_bytes(B, S, H)
    kk["attn_decode"] = entry(timed_calls(torch, sq, attn_fns(b)), b, "bytes")
    kk["attn_decode_split"] = entry(timed_calls(torch, sq, attn_fns(b, split=True)), b, "bytes")
    kk["attn_decode_split"]["workspace_bytes"] = sq.attn_decode_workspace_bytes(B, S, H, D)
    if variants:
        b = kv_bytes(E, bits=8)
        kk["kv_quant_8bit"] = entry(timed_calls(torch, sq, kv_fns(b, bits=8)), b, "bytes")
        b = kv_bytes(E)
        kk["kv_quant_clip95"] = entry(timed_calls(torch, sq, kv_fns(b, k_clip=0.95, v_clip=0.95)), b, "bytes")
        b = kv_bytes(E, param_bytes=2)
        kk["kv_quant_fp16_params"] = entry(timed_calls(torch, sq, kv_fns(b, param_dtype=torch.float16)), b, "bytes")
        b = attn_bytes(B, S, H, param_bytes=2)
        kk["attn_decode_fp16_params"] = entry(timed_calls(torch, sq, attn_fns(b, param_dtype=torch.float16)), b,
                                              "bytes")
    for n, e in kk.items():
        e["traffic"] = measured_traffic(f"c4/{n}")
    del q, k, v
    torch.cuda.empty_cache()
    return {"workload": workloads.R3_KV["name"], "kernels": kk}


def tiny_config(torch, sq, workloads, dev):
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    x, w = workloads.tiny_inputs()
    xg = up(x)
    wq = sq.pack_w4(up(w), None, 256)
    q = sq.had_quant_act(xg, None, 256)[:3]
    y = sq.w4a4_linear(*q, *wq)[0]
    t_q = timed_calls(torch, sq, [lambda: sq.had_quant_act(xg, None, 256, out=q)], reps=50)
    t_g = timed_calls(torch, sq, [lambda: sq.w4a4_linear(*q, *wq, out=y)], reps=50)
    M, K, N = x.shape[0], x.shape[1], w.shape[0]
    return {"workload": workloads.TINY["name"],
            "kernels": {"rot_quant": entry(t_q, had_bytes(M, K), "bytes", "latency"),
                        "gemm": entry(t_g, 2 * M * N * K, "ops", "latency")}}


def config_report(torch, sq, workloads, dev, only=None, variants=True):
    rep = {}
    if only in (None, "c1"):
        rep["c1_tiny"] = tiny_config(torch, sq, workloads, dev)
    if only in (None, "c2", "variants"):
        rep["c2_llama2_7b"] = mlp_config("c2", workloads.LLAMA2_7B_MLP, torch, sq, workloads, dev, variants)
    if only in (None, "c3", "variants"):
        rep["c3_llama3_8b"] = mlp_config("c3", workloads.LLAMA3_8B_MLP, torch, sq, workloads, dev, variants)
    if only in (None, "c4", "variants"):
        rep["c4_r3_kv"] = kv_config(torch, sq, workloads, dev, variants)
    if only in (None, "c5"):
        big = workloads.LLAMA2_70B_DECODE[-1]  # the three decode sizes share weights and row prefixes
        inp = workloads.mlp_inputs(big)
        for sh in workloads.LLAMA2_70B_DECODE:
            rep[f"c5_llama2_70b_m{sh.M}"] = mlp_config(f"c5m{sh.M}", big, torch, sq, workloads, dev, False,
                                                       inp=inp, tokens=sh.M)
        del inp
    return rep


# ---------------------------------------------------------------- CPU oracle baseline

def cpu_baseline(shape, target_s):
    """The oracle, as it stands, on a row slice of the chained step (rows are independent)."""
    import threadpoolctl

    from oracle import hadamard as ohad
    from oracle import kv as okv
    from oracle import linear as olin
    from paper_2405_16406_amd import workloads

    cores = len(os.sched_getaffinity(0))
    with threadpoolctl.threadpool_limits(cores):
        info = threadpoolctl.threadpool_info()
        threads = max([i.get("num_threads", 1) for i in info] or [1])
        full = workloads.mlp_inputs(shape, rows=1)
        ha = ohad.dense_factor(shape.had_dense)
        # offline weight preparation (not timed)
        wg = olin.pack_w4(full["w_gate"])
        wu = olin.pack_w4(full["w_up"])
        wd = olin.pack_w4(full["w_down"], ha, shape.had_pow2)

        def run(rows):
            inp = workloads.mlp_inputs(shape, rows=rows)
            q, k, v = (workloads.head_acts(workloads.rng_for(900), 1, rows, 32, 128, 2, 30.0) for _ in range(3))
            t0 = time.perf_counter()
            okv.qk_had_kvquant(q, k, v)
            _, a1, b1, _, qa1 = olin.had_quant_act(inp["x_in"], None, 1)
            hh, _, _ = olin.swiglu_linear(qa1, a1[:, 0], b1[:, 0], wg[3], wg[1], wg[2], wu[3], wu[1], wu[2])
            _, a2, b2, _, qa2 = olin.had_quant_act(hh, ha, shape.had_pow2)
            olin.w4a4_linear(qa2, a2[:, 0], b2[:, 0], wd[3], wd[1], wd[2])
            return time.perf_counter() - t0

        rows = 64
        dt = run(rows)
        while dt < target_s / 3 and rows < shape.M:
            rows = min(shape.M, rows * 4)
            dt = run(rows)
    ops = 3 * 2 * rows * shape.inter * shape.hidden
    return {"value": round(ops / dt / 1e12, 5), "unit": "TOPS", "cores": int(threads), "kind": "oracle",
            "sample": f"first {rows} of {shape.M} token rows of the same chained layer step (KV quant, act "
                      f"quant, gate/up with SiLU, R4 + quant, down; exact fp64-BLAS integer GEMM), {dt:.2f} s"}


# ---------------------------------------------------------------- profile summaries

# The rocprofv3 runs whose outputs --summarize reads (from /tmp with TMPDIR=/tmp; DIR =
# rocprofv3 output root).  Each part runs in a process of its own.
PARTS = ("step", "c3", "c4", "c5")
PROFILE_COMMANDS = {}
for _p in PARTS:
    PROFILE_COMMANDS[f"trace_{_p}"] = (f"rocprofv3 --kernel-trace --stats --output-format csv -d DIR/trace_{_p} -o run -- "
                                       f"python3 /root/repo/bench.py --only {_p} --no-cpu --steps 20")
    for _c in ("FETCH_SIZE", "WRITE_SIZE"):
        PROFILE_COMMANDS[f"pmc_{_c}_{_p}"] = (f"rocprofv3 --pmc {_c} --output-format csv -d DIR/pmc_{_c}_{_p} -o run -- "
                                              f"python3 /root/repo/bench.py --only {_p} --no-cpu --steps 5 --warmup 2")
for _c in ("FETCH_SIZE", "WRITE_SIZE"):
    PROFILE_COMMANDS[f"calib_{_c}"] = (f"rocprofv3 --pmc {_c} --output-format csv -d DIR/calib_{_c} -o run -- "
                                       f"python3 /root/repo/bench.py --calib-copy")
PROFILE_COMMANDS["summary"] = "python3 bench.py --summarize DIR"

SOURCE_OF = {"qk_had_kvquant": "kv_quant.hip", "quant_rows_identity": "had_quant.hip",
             "had_quant_act_generic": "had_quant.hip", "had_quant_": "had_quant_kron.hip",
             "w4a4_gemm": "w4a4_gemm.hip", "w4a4_gemv": "w4a4_gemm.hip", "attn_decode": "kv_attn.hip"}


def _csv_rows(d, pattern):
    import csv
    import glob
    out = []
    for f in sorted(glob.glob(os.path.join(d, pattern))):
        with open(f) as fh:
            out += list(csv.DictReader(fh))
    return out


def _short(name):
    name = name.replace("(anonymous namespace)::", "").replace("sq::", "")
    for cut in ("(sq::", "(RotQuantArgs", "(GemmArgs", "(KvArgs", "(AttnArgs", "(long", "(int"):
        if cut in name:
            name = name[:name.index(cut)]
    return name.replace("void ", "").strip()


def _pmc_per_kernel(rows, counter):
    """mean over dispatches of the counter summed over its dimensions, per (kernel, grid)"""
    per = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        key = (r["Kernel_Name"], int(r["Grid_Size"]), int(r["Dispatch_Id"]))
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    agg = {}
    for (name, grid, _), v in per.items():
        agg.setdefault((name, grid), []).append(v)
    return {k: (float(np.mean(v)), len(v)) for k, v in agg.items()}


def _source(name):
    for frag, src in SOURCE_OF.items():
        if frag in name:
            return src
    return None


def summarize(d):
    """Turn the rocprofv3 outputs of PROFILE_COMMANDS (DIR = d) into profiles/ summaries:
    per part a kernel-duration table and an HBM-traffic table, and hbm_traffic.json with
    the bytes per launch of every kernel (keyed part/kernel and by name and grid)."""
    os.makedirs(PROFILE_DIR, exist_ok=True)
    cf = _pmc_per_kernel(_csv_rows(d, "calib_FETCH_SIZE/*counter_collection.csv"), "FETCH_SIZE")
    cw = _pmc_per_kernel(_csv_rows(d, "calib_WRITE_SIZE/*counter_collection.csv"), "WRITE_SIZE")
    cfk = [v[0] for k, v in cf.items() if "probe_copy" in k[0]]
    cwk = [v[0] for k, v in cw.items() if "probe_copy" in k[0]]
    f_fetch = CALIB_BYTES / (cfk[0] * 1024.0)
    f_write = CALIB_BYTES / (cwk[0] * 1024.0)
    names = {"step": "LLaMA-2-7B layer step (M = 2048), chained", "c3": "LLaMA-3-8B MLP (M = 4096), isolated kernels",
             "c4": "R3 + KV cache [8, 2048, 32, 128] and decode attention, isolated kernels",
             "c5": "LLaMA-2-70B decode (M = 1, 8, 16), isolated kernels"}
    traffic = {"fetch_factor": f_fetch, "write_factor": f_write,
               "calibration": f"probe_copy of {CALIB_BYTES >> 20} MiB: FETCH_SIZE {cfk[0]:.0f} KiB, "
                              f"WRITE_SIZE {cwk[0]:.0f} KiB per dispatch",
               "commands": PROFILE_COMMANDS, "kernels": {}, "by_grid": {}}
    for part in PARTS:
        cmds = "\n".join(f"    {c.replace('DIR', '<DIR>')}" for k, c in PROFILE_COMMANDS.items()
                         if k.endswith("_" + part) or k.startswith("calib"))
        trace = _csv_rows(d, f"trace_{part}/*kernel_trace.csv")
        if not trace:
            continue
        dur = {}
        for r in trace:
            grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
            dur.setdefault((r["Kernel_Name"], grid), []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
        lines = [f"# Kernel durations: {names[part]}", "",
                 "rocprofv3 kernel trace of `bench.py --only " + part + "`; every launch of a kernel counts in",
                 "its row (warm-up, timed and per-kernel event passes).  Commands (from /tmp, TMPDIR=/tmp):", "",
                 cmds, "",
                 "The first launches of each kernel run on a cold chip (clock, caches); the median is the",
                 "steady state that bench.py's second, event-timed pass reports.", "",
                 "| kernel | grid (threads) | calls | avg us | median us | min us | max us |",
                 "|---|---:|---:|---:|---:|---:|---:|"]
        for (name, grid), v in sorted(dur.items(), key=lambda kv: -np.mean(kv[1]) * len(kv[1])):
            if "sq::" not in name:  # the library's kernels only (not torch's set-up copies)
                continue
            lines.append(f"| `{_short(name)}` | {grid} | {len(v)} | {np.mean(v):.1f} | {np.median(v):.1f} | "
                         f"{np.min(v):.1f} | {np.max(v):.1f} |")
        with open(os.path.join(PROFILE_DIR, f"kernel_stats_{part}.md"), "w") as f:
            f.write("\n".join(lines) + "\n")
        fetch = _pmc_per_kernel(_csv_rows(d, f"pmc_FETCH_SIZE_{part}/*counter_collection.csv"), "FETCH_SIZE")
        write = _pmc_per_kernel(_csv_rows(d, f"pmc_WRITE_SIZE_{part}/*counter_collection.csv"), "WRITE_SIZE")
        lines = [f"# HBM traffic per launch: {names[part]}", "",
                 "rocprofv3 FETCH_SIZE and WRITE_SIZE (KiB per dispatch, one counter per run), scaled by what",
                 f"the same counters read for the probe copy kernel: FETCH_SIZE reads {cfk[0]:.0f} KiB for "
                 f"{CALIB_BYTES >> 10} KiB read (factor {f_fetch:.4f}),",
                 f"WRITE_SIZE {cwk[0]:.0f} KiB for {CALIB_BYTES >> 10} KiB written (factor {f_write:.4f}).",
                 "Commands (from /tmp, TMPDIR=/tmp):", "", cmds, "",
                 "| kernel | grid (threads) | dispatches | FETCH KiB | WRITE KiB | HBM read MB | HBM write MB |",
                 "|---|---:|---:|---:|---:|---:|---:|"]
        for key in sorted(fetch, key=lambda k: -fetch[k][0]):
            if "sq::" not in key[0]:
                continue
            fk, n = fetch[key]
            wk = write.get(key, (float("nan"), 0))[0]
            rd, wr = fk * 1024 * f_fetch, wk * 1024 * f_write
            lines.append(f"| `{_short(key[0])}` | {key[1]} | {n} | {fk:.0f} | {wk:.0f} | {rd / 1e6:.2f} | "
                         f"{wr / 1e6:.2f} |")
            src = _source(key[0])
            if src and np.isfinite(wr):
                traffic["by_grid"][f"{part}|{_short(key[0])}|{key[1]}"] = {
                    "source": src, "source_sha256_16": source_hash(os.path.join(CSRC, src)),
                    "read_bytes": round(rd), "write_bytes": round(wr), "dispatches": n}
        with open(os.path.join(PROFILE_DIR, f"hbm_traffic_{part}.md"), "w") as f:
            f.write("\n".join(lines) + "\n")
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(traffic, f, indent=1)
    print(json.dumps({k: v for k, v in traffic.items() if k in ("fetch_factor", "write_factor")}))


# ---------------------------------------------------------------- main

def main():
    args = parse()
    if args.summarize:
        summarize(args.summarize)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "one GPU only: the rotated W4A4 path is not "
                                   "sharded across GPUs", "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2405_16406_amd import sq, workloads

    dev = torch.device("cuda:0")
    if args.calib_copy:
        pr = probe()
        src = torch.empty(CALIB_BYTES, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
        for _ in range(4):
            pr.check(pr.L.sq_probe_copy(ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr()),
                                        CALIB_BYTES, 2048, stream), "copy probe")
        torch.cuda.synchronize()
        print(json.dumps({"calib_copy_bytes": CALIB_BYTES, "launches": 4}), flush=True)
        return

    if args.only not in (None, "step"):
        t0 = time.perf_counter()
        res = measure_peaks(torch, dev) if args.only == "peaks" else \
            config_report(torch, sq, workloads, dev, only=args.only, variants=args.only == "variants")
        print(json.dumps({"only": args.only, "result": res, "wall_s": round(time.perf_counter() - t0, 1)}), flush=True)
        return

    st = run_step(args, torch, sq, workloads, dev)
    shape = st["shape"]
    M, HID, INTER = shape.M, shape.hidden, shape.inter
    value = st["step_ops"] / (st["ms_step"] * 1e-3) / 1e12
    dom = st["kernels"]["gate_up_swiglu"]
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(st["ms_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8",
        "data": "synthetic",
        "config": {"workload": "LLaMA-2-7B layer, M=2048 tokens, chained: R3+KV4 quant [1,2048,32,128]; "
                               "act quant [2048,4096]; gate/up W4A4 with SiLU(g)*u [2048x4096]x[2x11008x4096] "
                               "-> h; R4 H_172(x)S_64 + quant of h [2048,11008]; down W4A4 [2048x11008]x[4096x11008]",
                   "tokens": M, "hidden": HID, "intermediate": INTER, "heads": 32, "head_dim": 128,
                   "r4": f"H_{shape.had_dense} (x) S_{shape.had_pow2}", "buffer_sets": args.sets},
        # the dominant kernel: the gate/up product (two thirds of the step's ops)
        "roofline": {"kernel": "w4a4_gemm_ring (gate/up with SiLU)", "bound": "mfma", "achieved": dom["achieved"],
                     "peak": INT8_PEAK_TOPS, "unit": "TOP/s", "frac": dom["frac"],
                     "traffic": dom["traffic"]["total"] if dom["traffic"] else None,
                     "traffic_read_write": [dom["traffic"]["read"], dom["traffic"]["write"]] if dom["traffic"] else None,
                     "ops_per_launch": dom["ops"], "algorithmic_bytes_per_launch": dom["algorithmic_bytes"],
                     "us_per_launch": dom["us"]},
        "kernels": st["kernels"],
        "kernel_timing": "per kernel: mean over a second pass of the same K steps of the kernel's own "
                         "start/end HIP events (hipExtLaunchKernel); kernel_sum_ms is their sum; inside the step "
                         "h and the codes pass between kernels through HBM and the Infinity Cache",
        "kernel_sum_ms": round(sum(st["per"].values()), 4),
        "wall_s": round(st["wall"], 3),
    }
    if args.only is None and not args.no_configs:
        t0 = time.perf_counter()
        out["peaks"] = measure_peaks(torch, dev)
        out["configs"] = config_report(torch, sq, workloads, dev)
        out["configs_note"] = ("each kernel alone, cycling through copies of its operands (> 1 GB in all) so that "
                               "every launch reads HBM; mean of its own start/end events over >= 20 launches; "
                               "decode-sized GEMMs are weight streams (bound hbm)")
        out["configs_wall_s"] = round(time.perf_counter() - t0, 1)
    if not args.no_cpu and args.only is None:
        out["cpu_baseline"] = cpu_baseline(shape, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
