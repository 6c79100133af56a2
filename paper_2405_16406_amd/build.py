"""Builds libsq.so (HIP kernels for gfx950 + the C-ABI host code) and libsq_probe.so (the
roofline probes of include/sq_probe.h, used by the benchmark) in-tree with hipcc.

    python -m paper_2405_16406_amd.build        # compiles every source, always
    python -m paper_2405_16406_amd.build asan   # also the sanitizer build (below)

Objects go to _build/ at the repository root; the library is written next to this
file.  Compile flags:
  --offload-arch=gfx950           CDNA4 only
  -O3 -std=c++17
  -ffp-contract=off               no fused multiply-add contraction, so the quantizer's
                                  fp32 op sequence rounds after every step
  -Xclang -target-feature -Xclang -packed-fp32-ops
                                  no packed fp32 VALU instructions in the device code

Sanitizer build (build_sanitized): the host-only sources (argument validation, error
state, Hadamard construction) compiled with AddressSanitizer and UndefinedBehaviorSanitizer
(host code only: every -fsanitize= sits behind -Xarch_host), linked with the unchanged
kernel objects into _build/asan/libsq_asan.so.  A process loading it needs the shared
ASan runtime loaded first (asan_runtime() gives its path).
"""

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libsq.so")
PROBE_SRC = os.path.join(PKG, "probe", "roofline_probe.hip")
PROBE_LIB = os.path.join(PKG, "libsq_probe.so")
ASAN_DIR = os.path.join(BUILD_DIR, "asan")
ASAN_LIB = os.path.join(ASAN_DIR, "libsq_asan.so")

ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", "-ffp-contract=off", f"-I{INCLUDE}", f"-I{CSRC}"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-shared-libsan"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libsq.so)")


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))


def _compile(src: str, out_dir: str = BUILD_DIR, extra=()) -> str:
    obj = os.path.join(out_dir, os.path.basename(src) + ".o")
    cmd = [hipcc(), *COMMON, *DEVICE, *extra, "-c", src, "-o", obj]
    if src.endswith(".cpp"):
        cmd = [hipcc(), *COMMON, *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def _link(objs, out: str) -> None:
    tmp = out + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Wl,--no-undefined", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    """Compile every source, link libsq.so and libsq_probe.so; returns libsq.so's path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sources() + [PROBE_SRC]
    workers = min(len(srcs), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(workers) as ex:
        objs = list(ex.map(_compile, srcs))
    _link(objs[:-1], LIB)
    _link(objs[-1:], PROBE_LIB)
    if verbose:
        print(f"built {LIB} and {PROBE_LIB}")
    return LIB


def asan_runtime() -> str:
    """Path of the shared AddressSanitizer runtime of hipcc's clang."""
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "llvm", "bin", "clang++")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang++"
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError("shared ASan runtime not found")
    return path


def build_sanitized(verbose: bool = False) -> str:
    """Host sources with ASan + UBSan, kernels unchanged; returns the library path."""
    os.makedirs(ASAN_DIR, exist_ok=True)
    srcs = sources()
    host = [s for s in srcs if s.endswith(".cpp")]
    dev = [s for s in srcs if s.endswith(".hip")]
    workers = min(len(srcs), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(workers) as ex:
        objs = list(ex.map(lambda s: _compile(s, ASAN_DIR, SANITIZE), host))
        objs += list(ex.map(lambda s: _compile(s, ASAN_DIR), dev))
    tmp = ASAN_LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *SANITIZE, *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, ASAN_LIB)
    if verbose:
        print(f"built {ASAN_LIB}")
    return ASAN_LIB


if __name__ == "__main__":
    build(verbose=True)
    if len(sys.argv) > 1 and sys.argv[1] == "asan":
        build_sanitized(verbose=True)
    sys.exit(0)
