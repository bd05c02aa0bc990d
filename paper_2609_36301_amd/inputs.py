"""Seeded synthetic router inputs, shared by the HIP path's callers and the oracle.

This module draws random numbers and rounds them to bfloat16. It holds none of the
router's arithmetic: no projection, no logits, no selection, no softmax. Both the
tests (which feed the same arrays to the fp64 oracle and to the HIP library) and
`bench.py` take their inputs from here, so the two sides see identical bits.

Distributions follow the router setup of the paper: hidden states x ~ N(0, 1), the
down-projection R1 (h x r) ~ N(0, 1/h) and the expert matrix R2 (r x M) ~ N(0, 1/r).
With these variances z = x R1 has unit-variance entries and so do the logits z R2
(variance-matching lemma, Appendix "Initialization": Var = r s1^2 s2^2 |x|^2).

Arrays are returned as numpy uint16 holding bfloat16 bit patterns, in the
mathematical (row-major) orientation: x [T][h], R1 [h][r], R2 [r][M].  The HIP
library takes the two factors transposed (R1^T [r][h], R2^T [M][r]); callers make
those copies with `transposed_factors`.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "RouterInputs",
    "make_inputs",
    "f32_to_bf16_bits",
    "bf16_bits_to_f32",
    "transposed_factors",
    "make_workload_inputs",
]


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One router problem size plus the recipe for its synthetic inputs."""

    name: str
    T: int  # tokens routed per call
    h: int  # hidden size
    r: int  # router rank
    M: int  # experts
    k: int  # experts selected per token
    dup_token_frac: float = 0.0  # fraction of token rows overwritten by copies of other rows
    expert_bias_var: float = 0.0  # variance of a per-expert offset added to every entry of R2's column
    histogram: bool = False  # whether the per-expert histogram is part of the step
    description: str = ""


WORKLOADS: dict[str, Workload] = {
    w.name: w
    for w in (
        Workload("tiny", 256, 512, 16, 256, 8,
                 description="small parity case, oracle finishes in well under a second"),
        Workload("teaser_prefill", 16384, 512, 32, 4096, 8,
                 description="prefill at the scale of the paper's teaser layer (h=512)"),
        Workload("mid", 32768, 2048, 64, 16384, 8, dup_token_frac=0.05, histogram=True,
                 description="mid-size model; 5% duplicated tokens; expert histogram"),
        Workload("fine_grained", 16384, 4096, 64, 65536, 8, expert_bias_var=0.5, histogram=True,
                 description="fine-grained experts; skewed load from per-expert bias; histogram"),
        Workload("decode", 128, 4096, 64, 262144, 16,
                 description="decode-shaped batch with very many experts; R2 stream dominates"),
    )
}


# Shapes outside the benchmark suite, for timing routes the suite does not reach: the paper's
# rank sweeps go up to r = 256 (Section "Routing expressivity"); r = 128 takes the wide route.
EXTRA_WORKLOADS: dict[str, Workload] = {
    w.name: w
    for w in (
        Workload("rank128", 16384, 2048, 128, 16384, 8, histogram=True,
                 description="rank-sweep shape at r = 128 (wide route); expert histogram"),
    )
}


def find_workload(name: str) -> Workload:
    """A benchmark-suite workload or one of the extra shapes, by name."""
    return WORKLOADS[name] if name in WORKLOADS else EXTRA_WORKLOADS[name]


@dataclasses.dataclass
class RouterInputs:
    """bf16 bit patterns (uint16) in mathematical orientation."""

    x: np.ndarray  # [T][h]
    R1: np.ndarray  # [h][r]
    R2: np.ndarray  # [r][M]
    dup_dst: np.ndarray  # rows of x overwritten by copies (may be empty)
    dup_src: np.ndarray  # row each dup_dst row was copied from
    seed: int

    @property
    def shape(self):
        T, h = self.x.shape
        r, M = self.R2.shape
        return T, h, r, M


def make_inputs(T: int, h: int, r: int, M: int, *, seed: int = 0,
                dup_token_frac: float = 0.0, expert_bias_var: float = 0.0,
                dup_expert_frac: float = 0.0) -> RouterInputs:
    """Draw one seeded problem.

    Draw order from a single PCG64 stream: x, R1, R2, per-expert bias, duplicate-token map,
    duplicate-expert map.  Each tensor is drawn in float64, narrowed to float32, then rounded
    to bfloat16.  The per-expert bias b_e ~ N(0, expert_bias_var) is added to every entry of
    column e of R2 before rounding.  Duplicated tokens copy the *rounded* row, so they are
    bit-identical.  `dup_expert_frac` copies whole R2 columns onto other columns, which makes
    exact ties between experts (identical logits for every token).
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    x = f32_to_bf16_bits(rng.standard_normal((T, h)).astype(np.float32))
    R1 = f32_to_bf16_bits((rng.standard_normal((h, r)) * math.sqrt(1.0 / h)).astype(np.float32))
    R2f = rng.standard_normal((r, M)) * math.sqrt(1.0 / r)
    if expert_bias_var > 0.0:
        bias = rng.standard_normal(M) * math.sqrt(expert_bias_var)
        R2f = R2f + bias[None, :]
    R2 = f32_to_bf16_bits(R2f.astype(np.float32))
    dup_dst = np.zeros(0, dtype=np.int64)
    dup_src = np.zeros(0, dtype=np.int64)
    if dup_token_frac > 0.0 and T > 1:
        n = int(math.floor(dup_token_frac * T))
        if n > 0:
            dup_dst = np.sort(rng.choice(T, size=n, replace=False)).astype(np.int64)
            pool = np.setdiff1d(np.arange(T, dtype=np.int64), dup_dst)
            dup_src = rng.choice(pool, size=n, replace=True).astype(np.int64)
            x[dup_dst] = x[dup_src]
    if dup_expert_frac > 0.0 and M > 1:
        n = int(math.floor(dup_expert_frac * M))
        if n > 0:
            dst = rng.choice(M, size=n, replace=False)
            pool = np.setdiff1d(np.arange(M), dst)
            src = rng.choice(pool, size=n, replace=True)
            R2[:, dst] = R2[:, src]
    return RouterInputs(x=x, R1=R1, R2=R2, dup_dst=dup_dst, dup_src=dup_src, seed=seed)


def make_workload_inputs(w: Workload | str, *, seed: int = 0, T: int | None = None) -> RouterInputs:
    """Inputs for a named workload; `T` may shrink the token count (same h, r, M recipe)."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    return make_inputs(w.T if T is None else T, w.h, w.r, w.M, seed=seed,
                       dup_token_frac=w.dup_token_frac, expert_bias_var=w.expert_bias_var)


def transposed_factors(inp: RouterInputs) -> tuple[np.ndarray, np.ndarray]:
    """R1^T [r][h] and R2^T [M][r] as contiguous uint16 copies (the HIP library's layout)."""
    return np.ascontiguousarray(inp.R1.T), np.ascontiguousarray(inp.R2.T)
