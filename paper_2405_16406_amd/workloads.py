"""Seeded synthetic inputs with the shapes and value distributions of the paper's
LLaMA workloads (LLaMA-2 7B/70B, LLaMA-3 8B layers).

This module only draws random numbers; it holds none of the method's arithmetic.  It
is the one piece shared by the tests, the benchmark and the oracle checks, so that
both sides see byte-identical fp16 inputs.

Recipe (stand-in for the paper's WikiText2 / zero-shot activations and the LLaMA
weights, which are not available):
  * numpy PCG64 generator seeded with the workload's seed;
  * activations ~ N(0, 1) with a set of outlier channels, drawn once per tensor and
    shared by all rows, multiplied by a large factor (Sec. 2, Fig. 2 shows activation
    outliers concentrated in a few channels);
  * weights ~ N(0, 0.02^2);
  * everything is cast to fp16 (the paper's X_R is FP16, Sec. 2 eq. 1).
"""

from dataclasses import dataclass

import numpy as np


def rng_for(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def outlier_acts(rng: np.random.Generator, rows: int, cols: int, n_outlier: int,
                 scale: float) -> np.ndarray:
    """fp16 [rows, cols]: N(0,1) with n_outlier channels (columns) times scale."""
    x = rng.standard_normal((rows, cols), dtype=np.float32)
    if n_outlier:
        ch = rng.choice(cols, size=n_outlier, replace=False)
        x[:, ch] *= np.float32(scale)
    return x.astype(np.float16)


def weights(rng: np.random.Generator, rows: int, cols: int, std: float = 0.02) -> np.ndarray:
    """fp16 [rows, cols] ~ N(0, std^2)."""
    return (rng.standard_normal((rows, cols), dtype=np.float32) * np.float32(std)).astype(np.float16)


def head_acts(rng: np.random.Generator, B: int, S: int, H: int, D: int, n_outlier: int,
              scale: float) -> np.ndarray:
    """fp16 [B, S, H, D]: N(0,1) with n_outlier dims per head (same for all b, s) times scale."""
    x = rng.standard_normal((B, S, H, D), dtype=np.float32)
    for h in range(H):
        dims = rng.choice(D, size=n_outlier, replace=False)
        x[:, :, h, dims] *= np.float32(scale)
    return x.astype(np.float16)


@dataclass(frozen=True)
class MLPShape:
    """One LLaMA MLP layer at M tokens: gate/up [inter, hidden], down [hidden, inter].

    The down-projection input is rotated online by H_a (x) S_b with b = had_pow2,
    a = had_dense (a * b == inter).
    """
    name: str
    seed: int
    M: int
    hidden: int
    inter: int
    had_dense: int
    had_pow2: int

    @property
    def n_outlier_hidden(self) -> int:
        return int(round(0.01 * self.hidden))

    @property
    def n_outlier_inter(self) -> int:
        return int(round(0.01 * self.inter))


TINY = dict(name="tiny rotated W4A4 linear [16x256]x[256x256], Sylvester 256", seed=0,
            M=16, K=256, N=256, had_dense=1, had_pow2=256, n_outlier=4, scale=50.0)

LLAMA2_7B_MLP = MLPShape("LLaMA-2-7B MLP layer, M=2048", 1, 2048, 4096, 11008, 172, 64)
LLAMA3_8B_MLP = MLPShape("LLaMA-3-8B MLP layer, M=4096", 2, 4096, 4096, 14336, 28, 512)
LLAMA2_70B_DECODE = [MLPShape(f"LLaMA-2-70B MLP decode, M={m}", 4, m, 8192, 28672, 28, 1024)
                     for m in (1, 8, 16)]
R3_KV = dict(name="R3 + 4-bit KV cache, [8, 2048, 32, 128]", seed=3, B=8, S=2048, H=32, D=128,
             n_outlier=2, scale=30.0)


def tiny_inputs():
    """x fp16 [16, 256] with 4 outlier channels x50; w fp16 [256, 256] ~ N(0, 0.02^2)."""
    c = TINY
    rng = rng_for(c["seed"])
    x = outlier_acts(rng, c["M"], c["K"], c["n_outlier"], c["scale"])
    w = weights(rng, c["N"], c["K"])
    return x, w


def mlp_inputs(shape: MLPShape, rows: int | None = None):
    """Inputs of one MLP layer: dict with x_in [M, hidden], w_gate, w_up [inter, hidden],
    x_down [M, inter] (the down-projection input), w_down [hidden, inter].  All fp16.

    rows: generate only the first `rows` token rows of the activations (the weights are
    always whole).  Rows are drawn in the same order, so a prefix of rows equals the
    prefix of the full tensor.
    """
    m = shape.M if rows is None else rows
    rng_w = rng_for(1000 + shape.seed)
    w_gate = weights(rng_w, shape.inter, shape.hidden)
    w_up = weights(rng_w, shape.inter, shape.hidden)
    w_down = weights(rng_w, shape.hidden, shape.inter)
    x_in = _prefix_acts(shape.seed, 0, m, shape.hidden, shape.n_outlier_hidden)
    x_down = _prefix_acts(shape.seed, 1, m, shape.inter, shape.n_outlier_inter)
    return dict(x_in=x_in, w_gate=w_gate, w_up=w_up, x_down=x_down, w_down=w_down)


def _prefix_acts(seed: int, stream: int, rows: int, cols: int, n_outlier: int,
                 scale: float = 50.0) -> np.ndarray:
    """Outlier activations whose first r rows do not depend on how many rows are drawn."""
    rng_ch = rng_for(10_000 * seed + 2 * stream)
    ch = rng_ch.choice(cols, size=n_outlier, replace=False)
    out = np.empty((rows, cols), dtype=np.float16)
    rng = rng_for(10_000 * seed + 2 * stream + 1)
    blk = 256
    for r0 in range(0, rows, blk):
        r1 = min(rows, r0 + blk)
        x = rng.standard_normal((blk, cols), dtype=np.float32)[: r1 - r0]
        x[:, ch] *= np.float32(scale)
        out[r0:r1] = x.astype(np.float16)
    return out


def kv_inputs(B=None, S=None, H=None, D=None):
    """q, k, v fp16 [B, S, H, D] with 2 outlier dims per head x30 (R3_KV by default)."""
    c = R3_KV
    B = c["B"] if B is None else B
    S = c["S"] if S is None else S
    H = c["H"] if H is None else H
    D = c["D"] if D is None else D
    rng = rng_for(c["seed"])
    q = head_acts(rng, B, S, H, D, c["n_outlier"], c["scale"])
    k = head_acts(rng, B, S, H, D, c["n_outlier"], c["scale"])
    v = head_acts(rng, B, S, H, D, c["n_outlier"], c["scale"])
    return q, k, v
