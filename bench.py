"""Benchmark of the rotated W4A4 hot path on one MI355X.

One step = one pass of the whole path over one LLaMA-2-7B transformer layer's worth of
tokens (M = 2048):
  1. R3 + 4-bit KV quantization of Q, K, V [1, 2048, 32, 128]          sq_qk_had_kvquant
  2. per-token 4-bit quantization of the MLP input [2048, 4096]          sq_had_quant_act (identity)
  3. gate and up projections as one launch against the two packed weights
     stacked: [2048x4096] x [22016x4096]^T                               sq_w4a4_linear
  4. online R4 (H_172 (x) S_64) + 4-bit quantization of the down-projection
     input [2048, 11008]                                                 sq_had_quant_act
  5. down projection [2048x11008] x [4096x11008]^T                       sq_w4a4_linear
Weights are packed once beforehand (sq_pack_w4, R4 folded into W_down), as in
deployment; gate and up share the input, so their packed weights are stacked into one
[22016, 4096] matrix (packing is per output row, so this changes no code) and run as one
GEMM launch.  Inputs are synthetic (seeded, LLaMA-shaped, with outlier channels) and
already resident in HBM; eight input/weight sets (--sets) are rotated so that
consecutive steps do not hit the 256 MB Infinity Cache.

value = W4A4 linear ops of the step (3 x 2*M*N*K) / step time, in TOPS.  Per-kernel
durations come from a second pass over the same steps, in which the library attaches
a pair of HIP events to each kernel launch (start/stop of the launch itself, on the
stream the library runs on).  The CPU baseline times the oracle on a bounded slice of the same workload.

    python bench.py [--steps K] [--warmup W] [--no-cpu] [--report PATH]
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "W4A4 rotated-linear TOPS + Hadamard/quant GB/s at LLaMA-2-7B/3-8B shapes"
HBM_PEAK_GBS = 8000.0
INT8_PEAK_TOPS = 5000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=30)
    p.add_argument("--sets", type=int, default=8, help="input/weight sets rotated between steps")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU oracle time")
    p.add_argument("--report", default=None, help="write per-config kernel timings (JSON) here")
    p.add_argument("--calib-copy", action="store_true",
                   help="only run a plain 512 MiB device-to-device copy (counter calibration) and exit")
    p.add_argument("--summarize", default=None, metavar="DIR",
                   help="write the profiles/ summaries from rocprofv3 outputs under DIR and exit (no GPU)")
    return p.parse_args()


GEMM_SRC = os.path.join(ROOT, "paper_2405_16406_amd", "csrc", "w4a4_gemm.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "w4a4_gemm_llama2_7b_m2048_traffic.json")


def source_hash(path):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic():
    """HBM bytes per GEMM launch from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE runs, if
    they were taken on the current kernel source; otherwise None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256_16") != source_hash(GEMM_SRC):
        return None
    return t.get("bytes_per_launch")


PROFILE_DIR = os.path.join(ROOT, "profiles")
WORKLOAD_TAG = "llama2_7b_m2048"
# the commands whose outputs --summarize reads (run from /tmp with TMPDIR=/tmp; DIR = rocprofv3 output root)
PROFILE_COMMANDS = {
    "trace": "rocprofv3 --kernel-trace --stats --output-format csv -d DIR/trace -o bench -- "
             "python /root/repo/bench.py --no-cpu --steps 20",
    "fetch": "rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR/pmc_fetch -o bench -- "
             "python /root/repo/bench.py --no-cpu --steps 5 --warmup 2",
    "write": "rocprofv3 --pmc WRITE_SIZE --output-format csv -d DIR/pmc_write -o bench -- "
             "python /root/repo/bench.py --no-cpu --steps 5 --warmup 2",
    "calib_fetch": "rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR/pmc_cfetch -o copy -- "
                   "python /root/repo/bench.py --calib-copy",
    "calib_write": "rocprofv3 --pmc WRITE_SIZE --output-format csv -d DIR/pmc_cwrite -o copy -- "
                   "python /root/repo/bench.py --calib-copy",
    "summary": "python bench.py --summarize DIR",
}
REPORT_SPAN_BYTES = 1 << 30  # bytes each --report kernel cycles through
CALIB_BYTES = 512 << 20  # bytes read and written by each --calib-copy launch


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
    for cut in ("(sq::", "(RotQuantArgs", "(GemmArgs", "(KvArgs"):
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


def summarize(d):
    """Turn rocprofv3 outputs (the PROFILE_COMMANDS, DIR = d) into the profiles/ summaries."""
    cmds = "\n".join(f"    {c.replace('DIR', '<DIR>')}" for c in PROFILE_COMMANDS.values())
    os.makedirs(PROFILE_DIR, exist_ok=True)
    # ---- kernel durations
    trace = _csv_rows(d, "trace/*kernel_trace.csv")
    dur = {}
    for r in trace:
        grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
        key = (r["Kernel_Name"], grid)
        dur.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
    bench_line = ""
    bl = os.path.join(d, "trace_bench.json")
    if os.path.exists(bl):
        with open(bl) as f:
            bench_line = f.read().strip()
    lines = [f"# Kernel durations, rotated W4A4 path, LLaMA-2-7B layer (M = 2048 tokens)", "",
             "rocprofv3 kernel trace of the bench step: 30 warm-up steps, 20 timed steps, then the",
             "same 20 steps again with per-kernel timing events.  The 8 buffer sets are built once",
             "before them (torch roll + pack_w4).  Every launch of a kernel counts in its row.",
             "Commands (from /tmp, TMPDIR=/tmp):", "",
             cmds, "", "| kernel | grid (threads) | calls | avg us | min us | max us |",
             "|---|---:|---:|---:|---:|---:|"]
    for (name, grid), v in sorted(dur.items(), key=lambda kv: -np.mean(kv[1]) * len(kv[1])):
        lines.append(f"| `{_short(name)}` | {grid} | {len(v)} | {np.mean(v):.1f} | {np.min(v):.1f} | {np.max(v):.1f} |")
    if bench_line:
        lines += ["", "bench.py line printed by the traced run:", "", "```", bench_line, "```"]
    with open(os.path.join(PROFILE_DIR, f"rotated_w4a4_{WORKLOAD_TAG}_kernel_stats.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    # ---- HBM traffic from FETCH_SIZE / WRITE_SIZE, scaled by the copy calibration
    fetch = _pmc_per_kernel(_csv_rows(d, "pmc_fetch/*counter_collection.csv"), "FETCH_SIZE")
    write = _pmc_per_kernel(_csv_rows(d, "pmc_write/*counter_collection.csv"), "WRITE_SIZE")
    cf = _pmc_per_kernel(_csv_rows(d, "pmc_cfetch/*counter_collection.csv"), "FETCH_SIZE")
    cw = _pmc_per_kernel(_csv_rows(d, "pmc_cwrite/*counter_collection.csv"), "WRITE_SIZE")
    cfk = [v[0] for k, v in cf.items() if "copyBuffer" in k[0]]
    cwk = [v[0] for k, v in cw.items() if "copyBuffer" in k[0]]
    f_fetch = CALIB_BYTES / (cfk[0] * 1024.0)
    f_write = CALIB_BYTES / (cwk[0] * 1024.0)
    lines = [f"# HBM traffic per launch, rotated W4A4 path, LLaMA-2-7B layer (M = 2048 tokens)", "",
             "rocprofv3 FETCH_SIZE and WRITE_SIZE (KiB per dispatch, one counter per run), scaled by",
             "what the same counters read for a plain 512 MiB device-to-device copy:",
             f"FETCH_SIZE reads {cfk[0]:.0f} KiB for 524288 KiB read (factor {f_fetch:.4f}),",
             f"WRITE_SIZE reads {cwk[0]:.0f} KiB for 524288 KiB written (factor {f_write:.4f}).",
             "Commands (from /tmp, TMPDIR=/tmp):", "", cmds, "",
             "| kernel | grid (threads) | dispatches | FETCH KiB | WRITE KiB | HBM read MB | HBM write MB |",
             "|---|---:|---:|---:|---:|---:|---:|"]
    gemm = []
    for key in sorted(fetch, key=lambda k: -fetch[k][0]):
        fk, n = fetch[key]
        wk = write.get(key, (float("nan"), 0))[0]
        rd, wr = fk * 1024 * f_fetch, wk * 1024 * f_write
        lines.append(f"| `{_short(key[0])}` | {key[1]} | {n} | {fk:.0f} | {wk:.0f} | {rd / 1e6:.1f} | {wr / 1e6:.1f} |")
        if "w4a4_gemm" in key[0]:
            gemm += [(rd, wr)] * n
    with open(os.path.join(PROFILE_DIR, f"rotated_w4a4_{WORKLOAD_TAG}_hbm_traffic.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    t = {"kernel": "w4a4_gemm", "workload": "LLaMA-2-7B layer, M = 2048: gate, up and down projections",
         "kernel_source_sha256_16": source_hash(GEMM_SRC),
         "bytes_per_launch": round(float(np.mean([a + b for a, b in gemm]))),
         "read_bytes_per_launch": round(float(np.mean([a for a, _ in gemm]))),
         "write_bytes_per_launch": round(float(np.mean([b for _, b in gemm]))),
         "fetch_factor": f_fetch, "write_factor": f_write, "commands": PROFILE_COMMANDS}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(t, f, indent=1)
    print(json.dumps({k: t[k] for k in ("bytes_per_launch", "read_bytes_per_launch", "write_bytes_per_launch")}))


def gemm_bytes(M, N, K):
    return M * K // 2 + N * K // 2 + 2 * M * N + 8 * (M + N)


def had_bytes(M, K, groups_per_row=1):
    return 2 * M * K + M * K // 2 + 8 * M * groups_per_row


def attn_bytes(B, S, H, D=128):
    """Decode attention over a 4-bit cache: K and V codes (D/2 bytes) and their fp32 alpha,
    beta per cached (token, head), plus the fp16 query and output per head."""
    return B * S * H * (2 * (D // 2) + 4 * 4) + 2 * B * H * D * 2


def kv_bytes(E):
    return 3 * 2 * E + 2 * E + 2 * (E // 2) + 2 * 8 * (E // 128)


def main():
    args = parse()
    if args.summarize:
        summarize(args.summarize)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this build runs on one GPU only: the rotated W4A4 path is not "
                                   "sharded across GPUs", "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2405_16406_amd import sq, workloads

    dev = torch.device("cuda:0")
    if args.calib_copy:
        src = torch.empty(512 << 20, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calib_copy_bytes": src.numel(), "launches": 4}), flush=True)
        return
    shape = workloads.LLAMA2_7B_MLP
    M, HID, INTER = shape.M, shape.hidden, shape.inter
    A, B = shape.had_dense, shape.had_pow2
    NH, HD = 32, 128

    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    had = up(sq.hadamard_factor(A))

    # ---- resident inputs: `sets` distinct sets of activations and packed weights, so that
    # consecutive steps do not find the previous step's data in the caches.  Set 0 comes from
    # the seeded generators; set s > 0 is set 0 with its rows rotated by s * 997 (tokens for
    # activations, output channels for weights): same distributions, different buffers.
    inp = workloads.mlp_inputs(shape)
    rng = workloads.rng_for(500)
    base = dict(x_in=up(inp["x_in"]), x_down=up(inp["x_down"]),
                qkv=[up(workloads.head_acts(rng, 1, M, NH, HD, 2, 30.0)) for _ in range(3)],
                w_gu=up(np.concatenate([inp["w_gate"], inp["w_up"]])), w_down=up(inp["w_down"]))
    del inp
    sets = []
    for s in range(args.sets):
        r = lambda t, dim=0: torch.roll(t, shifts=s * 997, dims=dim).contiguous()
        sets.append(dict(x_in=r(base["x_in"]), x_down=r(base["x_down"]), qkv=[r(t, 1) for t in base["qkv"]],
                         wgu=sq.pack_w4(r(base["w_gu"])),  # stacked gate/up rows
                         wd=sq.pack_w4(r(base["w_down"]), had, B)))
    del base
    torch.cuda.synchronize()

    # ---- outputs (shared by all sets)
    kv_out = dict(q_rot=torch.empty((1, M, NH, HD), dtype=torch.float16, device=dev),
                  k_q=torch.empty((1, M, NH, HD // 2), dtype=torch.uint8, device=dev),
                  k_alpha=torch.empty((1, M, NH, 1), dtype=torch.float32, device=dev),
                  k_beta=torch.empty((1, M, NH, 1), dtype=torch.float32, device=dev),
                  v_q=torch.empty((1, M, NH, HD // 2), dtype=torch.uint8, device=dev),
                  v_alpha=torch.empty((1, M, NH, 1), dtype=torch.float32, device=dev),
                  v_beta=torch.empty((1, M, NH, 1), dtype=torch.float32, device=dev))
    xq_in = (torch.empty((M, HID // 2), dtype=torch.uint8, device=dev),
             torch.empty((M, 1), dtype=torch.float32, device=dev),
             torch.empty((M, 1), dtype=torch.float32, device=dev))
    xq_dn = (torch.empty((M, INTER // 2), dtype=torch.uint8, device=dev),
             torch.empty((M, 1), dtype=torch.float32, device=dev),
             torch.empty((M, 1), dtype=torch.float32, device=dev))
    y_gu = torch.empty((M, 2 * INTER), dtype=torch.float16, device=dev)  # [gate | up]
    y_dn = torch.empty((M, HID), dtype=torch.float16, device=dev)

    names = ["kv_quant", "act_quant", "gate_up_gemm", "r4_had_quant", "down_gemm"]

    def calls(s):
        d = sets[s]
        return [
            lambda: sq.qk_had_kvquant(*d["qkv"], out=kv_out),
            lambda: sq.had_quant_act(d["x_in"], out=xq_in),
            lambda: sq.w4a4_linear(*xq_in, *d["wgu"], out=y_gu),
            lambda: sq.had_quant_act(d["x_down"], had, B, out=xq_dn),
            lambda: sq.w4a4_linear(*xq_dn, *d["wd"], out=y_dn),
        ]

    step_calls = [calls(s) for s in range(args.sets)]

    def step(s):
        for c in step_calls[s]:
            c()

    for w in range(args.warmup):
        step(w % args.sets)
    torch.cuda.synchronize()

    # ---- timed region: K whole steps back to back, nothing recorded between kernels
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
    ms_total = t_start.elapsed_time(t_end)
    ms_step = ms_total / args.steps

    # ---- per-kernel durations inside the step: the same K steps again, each call timed by
    # a pair of HIP events that the library attaches to its own kernel launch on the
    # launch stream (sq_time_next_call: kernel start and end, no marker packets between
    # kernels).  This pass is kept out of the timed region above: arming the events costs
    # host time per call and a few microseconds per kernel on the device.
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
    step_ops = 3 * gemm_ops
    value = step_ops / (ms_step * 1e-3) / 1e12
    # the two GEMM launches of a step: gate+up (2 x gemm_ops) and down (gemm_ops)
    gemm_ms = per["gate_up_gemm"] + per["down_gemm"]
    gemm_tops = step_ops / (gemm_ms * 1e-3) / 1e12
    E = M * NH * HD
    kernels = {
        "kv_quant": dict(ms=per["kv_quant"], GBps=kv_bytes(E) / (per["kv_quant"] * 1e-3) / 1e9),
        "act_quant": dict(ms=per["act_quant"], GBps=had_bytes(M, HID) / (per["act_quant"] * 1e-3) / 1e9),
        "r4_had_quant": dict(ms=per["r4_had_quant"], GBps=had_bytes(M, INTER) / (per["r4_had_quant"] * 1e-3) / 1e9),
    }
    kernels["gate_up_gemm"] = dict(ms=per["gate_up_gemm"], TOPS=2 * gemm_ops / (per["gate_up_gemm"] * 1e-3) / 1e12)
    kernels["down_gemm"] = dict(ms=per["down_gemm"], TOPS=gemm_ops / (per["down_gemm"] * 1e-3) / 1e12)
    for k_ in kernels.values():
        for f in list(k_):
            k_[f] = round(k_[f], 4)

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8",
        "data": "synthetic",
        "config": {"workload": "LLaMA-2-7B layer, M=2048 tokens: R3+KV4 quant [1,2048,32,128]; "
                               "act quant [2048,4096]; gate+up W4A4 [2048x4096]x[22016x4096] (stacked); "
                               "R4 H_172(x)S_64 + quant [2048,11008]; down W4A4 [2048x11008]x[4096x11008]",
                   "tokens": M, "hidden": HID, "intermediate": INTER, "heads": NH, "head_dim": HD,
                   "r4": f"H_{A} (x) S_{B}", "buffer_sets": args.sets},
        # w4a4_gemm: the step's two launches (gate+up, down); achieved = their ops / their time
        "roofline": {"kernel": "w4a4_gemm", "bound": "mfma", "achieved": round(gemm_tops, 2),
                     "peak": INT8_PEAK_TOPS, "unit": "TOP/s", "frac": round(gemm_tops / INT8_PEAK_TOPS, 4),
                     "traffic": measured_traffic(),
                     "ops_per_launch": step_ops // 2,
                     "algorithmic_bytes_per_launch": round((gemm_bytes(M, 2 * INTER, HID) + gemm_bytes(M, HID, INTER)) / 2)},
        "kernels": kernels,
        "kernel_timing": "per kernel: mean over a second pass of the same K steps of the kernel's own "
                         "start/end HIP events (hipExtLaunchKernel); kernel_sum_ms is their sum",
        "kernel_sum_ms": round(sum(per.values()), 4),
        "wall_s": round(wall, 3),
    }

    if args.report:
        out["report"] = args.report
        report = kernel_report(torch, sq, workloads, dev)
        with open(args.report, "w") as f:
            json.dump(report, f, indent=1)

    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(shape, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def cpu_baseline(shape, target_s):
    """The oracle, as it stands, on a row slice of the same workload (rows are independent)."""
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
            olin.w4a4_linear(qa1, a1[:, 0], b1[:, 0], wg[3], wg[1], wg[2])
            olin.w4a4_linear(qa1, a1[:, 0], b1[:, 0], wu[3], wu[1], wu[2])
            _, a2, b2, _, qa2 = olin.had_quant_act(inp["x_down"], ha, shape.had_pow2)
            olin.w4a4_linear(qa2, a2[:, 0], b2[:, 0], wd[3], wd[1], wd[2])
            return time.perf_counter() - t0

        rows = 64
        dt = run(rows)
        while dt < target_s / 3 and rows < shape.M:
            rows = min(shape.M, rows * 4)
            dt = run(rows)
    ops = 3 * 2 * rows * shape.inter * shape.hidden
    return {"value": round(ops / dt / 1e12, 5), "unit": "TOPS", "cores": int(threads), "kind": "oracle",
            "sample": f"first {rows} of {shape.M} token rows of the same layer (KV quant, act quant, gate/up, "
                      f"R4 + quant, down; exact fp64-BLAS integer GEMM), {dt:.2f} s"}


def kernel_report(torch, sq, workloads, dev):
    """Per-config kernel timings (each launch's own HIP events) for the docs.

    Each kernel cycles through enough copies of its inputs and outputs that they add up to
    more than the GPU's caches (256 MB of Infinity Cache, 4 MB of L2 per XCD), so repeated
    launches read HBM as a single pass would, not the previous launch's cached bytes.
    """
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    def n_copies(nbytes):
        return int(min(32, max(2, -(-REPORT_SPAN_BYTES // max(nbytes, 1)))))

    def timed(fns, reps=None):
        """Mean kernel time per launch over back-to-back launches: each call's own start/end
        events (sq_time_next_call), so neither host gaps nor launch overhead count."""
        reps = reps or max(20, 2 * len(fns))
        for f in fns:
            f()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for r in range(reps):
            sq.time_next_call(*evs[r])
            fns[r % len(fns)]()
        torch.cuda.synchronize()
        return sum(a.elapsed_time(b) for a, b in evs) / reps

    def act_fns(x, had, pow2, nbytes, bits=4, **var):
        """had_quant_act launches over distinct copies of x and of the outputs (var: clip,
        signs of the _ex entry point)."""
        fns = []
        for _ in range(n_copies(nbytes)):
            xc = x.clone()
            o = sq.had_quant_act(xc, had, pow2, bits=bits, **var)[:3]
            fns.append(lambda xc=xc, o=o: sq.had_quant_act(xc, had, pow2, bits=bits, out=o, **var))
        return fns

    def gemm8_fns(qx, w, nbytes):
        """w4a8_linear launches over distinct copies of the operands and of y."""
        fns = []
        for _ in range(n_copies(nbytes)):
            qc = tuple(t.clone() for t in qx)
            wc = tuple(t.clone() for t in w)
            y = sq.w4a8_linear(*qc, *wc)[0]
            fns.append(lambda qc=qc, wc=wc, y=y: sq.w4a8_linear(*qc, *wc, out=y))
        return fns

    def gemm_fns(qx, w, nbytes, swiglu=False):
        """w4a4_linear (or w4a4_linear_swiglu) launches over distinct copies of the operands
        and of the output."""
        fns = []
        for _ in range(n_copies(nbytes)):
            qc = tuple(t.clone() for t in qx)
            wc = tuple(t.clone() for t in w)
            if swiglu:
                y = sq.w4a4_linear_swiglu(*qc, *wc)
                fns.append(lambda qc=qc, wc=wc, y=y: sq.w4a4_linear_swiglu(*qc, *wc, out=y))
            else:
                y = sq.w4a4_linear(*qc, *wc)[0]
                fns.append(lambda qc=qc, wc=wc, y=y: sq.w4a4_linear(*qc, *wc, out=y))
        return fns

    rep = []
    cfgs = [workloads.LLAMA2_7B_MLP, workloads.LLAMA3_8B_MLP] + workloads.LLAMA2_70B_DECODE
    for sh in cfgs:
        inp = workloads.mlp_inputs(sh)
        had = up(sq.hadamard_factor(sh.had_dense))
        xin, xdn = up(inp["x_in"]), up(inp["x_down"])
        wg = sq.pack_w4(up(inp["w_gate"]))
        wgu = sq.pack_w4(up(np.concatenate([inp["w_gate"], inp["w_up"]])))
        wsw = sq.pack_w4(sq.interleave_gate_up(up(inp["w_gate"]), up(inp["w_up"])).contiguous())
        wd = sq.pack_w4(up(inp["w_down"]), had, sh.had_pow2)
        qi = sq.had_quant_act(xin)[:3]
        qd = sq.had_quant_act(xdn, had, sh.had_pow2)[:3]
        M, H, I = sh.M, sh.hidden, sh.inter
        b_aq, b_hq = had_bytes(M, H), had_bytes(M, I)
        b_g, b_gu, b_d = gemm_bytes(M, I, H), gemm_bytes(M, 2 * I, H), gemm_bytes(M, H, I)
        b_sw = b_gu - 2 * M * I  # half the output: fp16 [M, I]
        t_aq = timed(act_fns(xin, None, 1, b_aq))
        t_hq = timed(act_fns(xdn, had, sh.had_pow2, b_hq))
        t_g = timed(gemm_fns(qi, wg, b_g))
        t_gu = timed(gemm_fns(qi, wgu, b_gu))
        t_sw = timed(gemm_fns(qi, wsw, b_sw, swiglu=True))
        t_d = timed(gemm_fns(qd, wd, b_d))
        # W4A8: 8-bit activation codes (one byte each) into the same weights
        qi8 = sq.had_quant_act(xin, bits=8)[:3]
        qd8 = sq.had_quant_act(xdn, had, sh.had_pow2, bits=8)[:3]
        b8_aq, b8_hq = had_bytes(M, H) + M * H // 2, had_bytes(M, I) + M * I // 2
        b8_gu, b8_d = gemm_bytes(M, 2 * I, H) + M * H // 2, gemm_bytes(M, H, I) + M * I // 2
        t8_aq = timed(act_fns(xin, None, 1, b8_aq, bits=8))
        t8_hq = timed(act_fns(xdn, had, sh.had_pow2, b8_hq, bits=8))
        t8_gu = timed(gemm8_fns(qi8, wgu, b8_gu))
        t8_d = timed(gemm8_fns(qd8, wd, b8_d))
        # the variants: random-sign Hadamard S H with a clipped range (S adds K bytes per row
        # set, read from cache; not counted)
        sgn = up(np.where(workloads.rng_for(7).random(I) < 0.5, -1, 1).astype(np.int8))
        tv_hq = timed(act_fns(xdn, had, sh.had_pow2, b_hq, signs=sgn, clip=0.9))
        rep.append(dict(config=sh.name,
                        act_quant=dict(ms=t_aq, GBps=b_aq / t_aq / 1e6),
                        r4_had_quant=dict(ms=t_hq, GBps=b_hq / t_hq / 1e6),
                        r4_had_quant_signs_clip=dict(ms=tv_hq, GBps=b_hq / tv_hq / 1e6),
                        gate_gemm=dict(ms=t_g, TOPS=2 * M * I * H / t_g / 1e9, GBps=b_g / t_g / 1e6),
                        gate_up_gemm=dict(ms=t_gu, TOPS=4 * M * I * H / t_gu / 1e9, GBps=b_gu / t_gu / 1e6),
                        gate_up_swiglu_gemm=dict(ms=t_sw, TOPS=4 * M * I * H / t_sw / 1e9, GBps=b_sw / t_sw / 1e6),
                        down_gemm=dict(ms=t_d, TOPS=2 * M * I * H / t_d / 1e9, GBps=b_d / t_d / 1e6),
                        act_quant_8bit=dict(ms=t8_aq, GBps=b8_aq / t8_aq / 1e6),
                        r4_had_quant_8bit=dict(ms=t8_hq, GBps=b8_hq / t8_hq / 1e6),
                        gate_up_w4a8=dict(ms=t8_gu, TOPS=4 * M * I * H / t8_gu / 1e9, GBps=b8_gu / t8_gu / 1e6),
                        down_w4a8=dict(ms=t8_d, TOPS=2 * M * I * H / t8_d / 1e9, GBps=b8_d / t8_d / 1e6)))
        del inp, xin, xdn, wg, wgu, wsw, wd, qi, qd, qi8, qd8, sgn
        torch.cuda.empty_cache()
    q, k, v = (up(t) for t in workloads.kv_inputs())
    E = q.numel()
    fns = []
    for _ in range(n_copies(kv_bytes(E))):
        qc, kc, vc = q.clone(), k.clone(), v.clone()
        o = sq.qk_had_kvquant(qc, kc, vc)
        o.pop("k_rot")
        fns.append(lambda qc=qc, kc=kc, vc=vc, o=o: sq.qk_had_kvquant(qc, kc, vc, out=o))
    t_kv = timed(fns)
    fns = []
    for _ in range(n_copies(kv_bytes(E) * 3 // 2)):
        qc, kc, vc = q.clone(), k.clone(), v.clone()
        o = sq.qk_had_kvquant(qc, kc, vc, bits=8)
        o.pop("k_rot")
        fns.append(lambda qc=qc, kc=kc, vc=vc, o=o: sq.qk_had_kvquant(qc, kc, vc, out=o, bits=8))
    t_kv8 = timed(fns)
    fns = []
    for _ in range(n_copies(kv_bytes(E))):
        qc, kc, vc = q.clone(), k.clone(), v.clone()
        o = sq.qk_had_kvquant(qc, kc, vc, k_clip=0.95, v_clip=0.95)
        o.pop("k_rot")
        fns.append(lambda qc=qc, kc=kc, vc=vc, o=o: sq.qk_had_kvquant(qc, kc, vc, out=o, k_clip=0.95, v_clip=0.95))
    t_kvc = timed(fns)
    fns = []
    for _ in range(n_copies(kv_bytes(E))):
        qc, kc, vc = q.clone(), k.clone(), v.clone()
        o = sq.qk_had_kvquant(qc, kc, vc, param_dtype=torch.float16)
        o.pop("k_rot")
        fns.append(lambda qc=qc, kc=kc, vc=vc, o=o: sq.qk_had_kvquant(qc, kc, vc, out=o, param_dtype=torch.float16))
    t_kvh = timed(fns)
    b_kvh = kv_bytes(E) - 8 * (E // 128)  # 2 x 4 bytes fewer per group
    b_kv8 = kv_bytes(E) + E  # codes of K and V: one byte per element instead of half
    # decode attention of the last token's rotated query over that cache
    B, S, H, D = q.shape
    b_at = attn_bytes(B, S, H)
    fns = []
    for _ in range(n_copies(b_at)):
        qc, kc, vc = q.clone(), k.clone(), v.clone()
        o = sq.qk_had_kvquant(qc, kc, vc)
        qr = o["q_rot"][:, -1].contiguous()
        oa = torch.empty_like(qr)
        cache = (o["k_q"], o["k_alpha"], o["k_beta"], o["v_q"], o["v_alpha"], o["v_beta"])
        fns.append(lambda qr=qr, cache=cache, oa=oa: sq.attn_decode_kv4(qr, *cache, out=oa))
        del qc, kc, vc
    t_at = timed(fns)
    b_ath = b_at - B * S * H * 8  # fp16 group parameters
    fns = []
    for _ in range(n_copies(b_ath)):
        qc, kc, vc = q.clone(), k.clone(), v.clone()
        o = sq.qk_had_kvquant(qc, kc, vc, param_dtype=torch.float16)
        qr = o["q_rot"][:, -1].contiguous()
        oa = torch.empty_like(qr)
        cache = (o["k_q"], o["k_alpha"], o["k_beta"], o["v_q"], o["v_alpha"], o["v_beta"])
        fns.append(lambda qr=qr, cache=cache, oa=oa: sq.attn_decode_kv4(qr, *cache, out=oa))
        del qc, kc, vc
    t_ath = timed(fns)
    rep.append(dict(config=workloads.R3_KV["name"], kv_quant=dict(ms=t_kv, GBps=kv_bytes(E) / t_kv / 1e6),
                    kv_quant_8bit=dict(ms=t_kv8, GBps=b_kv8 / t_kv8 / 1e6),
                    kv_quant_clip95=dict(ms=t_kvc, GBps=kv_bytes(E) / t_kvc / 1e6),
                    kv_quant_fp16_params=dict(ms=t_kvh, GBps=b_kvh / t_kvh / 1e6),
                    attn_decode=dict(ms=t_at, GBps=b_at / t_at / 1e6),
                    attn_decode_fp16_params=dict(ms=t_ath, GBps=b_ath / t_ath / 1e6)))
    return rep


if __name__ == "__main__":
    main()
