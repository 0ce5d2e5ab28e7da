"""Seeded synthetic inputs for the fused W8A8 linear.

This module draws the bf16 activations X [M,K], weights W [N,K] and bias b [N] that
stand in for a diffusion transformer's linear-layer operands. It holds none of the
method's arithmetic (no quantization, no product, no epilogue): it only draws random
numbers and rounds them once to bf16. Both the CPU oracle's tests and the HIP path's
tests and benchmark take their inputs from here, so the two sides see the same bits.

Recipe (all draws in float32 from numpy's PCG64, then rounded to bf16 with
round-to-nearest-even by torch's dtype conversion):
  * X ~ N(0, 1) with two fixed outlier input channels multiplied by 20, at channels
    17 and 3K/4 + 5 (the activation-outlier pattern SmoothQuant-style W8A8 recipes are
    built for, Section 2 "W8A8 PTQ recipe and outliers").
  * "gelu" X: exact-erf GELU of N(0, 1), no outlier channels (the input of an MLP
    down-projection). The GELU here (scipy's erf) only shapes the distribution;
    neither the oracle nor the HIP path uses it.
  * "preact" X: N(0, 1), no outlier channels: the pre-activation of that MLP, drawn
    from the same numbers as "gelu" (same seed, same draw), for the path that applies
    GELU inside the quantizer.
  * "student_t" X: Student-t with 3 degrees of freedom, no outlier channels
    (heavy-tailed activations).
  * W ~ N(0, 0.02) times a per-output-channel multiplier drawn from U(0.5, 2).
  * b ~ N(0, 0.01).
The seed of a workload shape is 20260 + 100 * config + shape index.

The shapes are the hidden-size-4096 DiT family: 768px-like sequences have
M = 2304 image + 256 text = 2560 tokens, 1024px-like ones M = 4096 + 512 = 4608.
The paper's own model uses hidden size 4608 (Section 3, "Target architecture"); its
prompt sets and weights are private, so these synthetic tensors stand in for them.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = ["Shape", "WORKLOADS", "PAPER_SHAPES", "PAPER_M", "paper_shape", "make_inputs",
           "workload", "shape_seed", "bf16_bits_from_f32"]


@dataclasses.dataclass(frozen=True)
class Shape:
    name: str
    M: int
    K: int
    N: int
    dist: str = "outlier"      # "outlier" | "gelu" | "preact" | "student_t"
    seed: int = 0

    @property
    def ops(self) -> int:
        """Integer operations of the product (2 per multiply-accumulate)."""
        return 2 * self.M * self.N * self.K


def shape_seed(config: int, index: int) -> int:
    return 20260 + 100 * config + index


def _mk(config: int, entries):
    out = []
    for i, e in enumerate(entries):
        name, M, K, N = e[:4]
        dist = e[4] if len(e) > 4 else "outlier"
        out.append(Shape(name, M, K, N, dist, shape_seed(config, i)))
    return out


# Workloads: config index -> list of shapes.
WORKLOADS = {
    0: _mk(0, [("tiny", 64, 256, 128)]),
    1: _mk(1, [("attn_proj", 2560, 4096, 4096),
               ("qkv", 2560, 4096, 12288)]),
    2: _mk(2, [("mlp_up", 2560, 4096, 16384),
               ("mlp_down", 2560, 16384, 4096, "gelu")]),
    3: _mk(3, [("qkv", 4608, 4096, 12288),
               ("attn_out", 4608, 4096, 4096),
               ("mlp_up", 4608, 4096, 16384),
               ("mlp_down", 4608, 16384, 4096)]),
    4: _mk(4, [(f"m{M}_n{N}", M, 4096, N, "student_t")
               for M in (1, 77, 333, 4625) for N in (4096, 16384)]
           + [(f"m{M}_k3136", M, 3136, 4096, "student_t") for M in (1, 77, 333, 4625)]),
}


# The paper's own model: five distinct GEMM shapes (name, N, K) of its 4608-wide DiT
# (Section 3, "Target architecture"), timed over the token counts of its speedup claim,
# M = 512 .. 16384, which contain the in-model M ~ 4110 at 1024px (Section 5, "The
# kernel is exact and the GEMMs are compute-bound"). The down-projection reads a GELU
# output, the others outlier-channel activations.
PAPER_SHAPES = [("qkv", 13824, 4608), ("attn_out", 4608, 4608), ("ffn_up", 12288, 4608),
                ("ffn_down", 4608, 12288), ("llm_proj", 4608, 53248)]
PAPER_M = [512, 1024, 2048, 4096, 4110, 8192, 16384]


def paper_shape(name: str, M: int) -> Shape:
    """The paper shape `name` at M tokens (seed 20260 + 500 + 10 * shape + M index, M
    indexed in PAPER_M or appended after it)."""
    names = [p[0] for p in PAPER_SHAPES]
    i = names.index(name)
    _, N, K = PAPER_SHAPES[i]
    j = PAPER_M.index(M) if M in PAPER_M else len(PAPER_M)
    return Shape(name, M, K, N, "gelu" if name == "ffn_down" else "outlier",
                 shape_seed(5, 10 * i + j))


def workload(config: int, name: str) -> Shape:
    for s in WORKLOADS[config]:
        if s.name == name:
            return s
    raise KeyError(f"config {config} has no shape {name!r}")


def bf16_bits_from_f32(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest-even) and return the raw uint16 bits.

    The rounding is torch's float32 -> bfloat16 dtype conversion, an independent
    library routine (the oracle carries its own, written from the IEEE definition)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def _erf_gelu(z: np.ndarray) -> np.ndarray:
    import scipy.special
    return (0.5 * z * (1.0 + scipy.special.erf(z / math.sqrt(2.0)))).astype(np.float32)


def draw_x(rng: np.random.Generator, M: int, K: int, dist: str) -> np.ndarray:
    if dist == "outlier":
        x = rng.standard_normal((M, K), dtype=np.float32)
        for c in sorted({17, 3 * K // 4 + 5}):
            if c < K:
                x[:, c] *= np.float32(20.0)
    elif dist == "gelu":
        x = _erf_gelu(rng.standard_normal((M, K), dtype=np.float32))
    elif dist == "preact":
        x = rng.standard_normal((M, K), dtype=np.float32)
    elif dist == "student_t":
        x = rng.standard_t(3, size=(M, K)).astype(np.float32)
    else:
        raise ValueError(dist)
    return x


def draw_w(rng: np.random.Generator, N: int, K: int) -> np.ndarray:
    w = rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.02)
    mult = rng.uniform(0.5, 2.0, size=(N, 1)).astype(np.float32)
    return w * mult


def draw_b(rng: np.random.Generator, N: int) -> np.ndarray:
    return rng.standard_normal(N, dtype=np.float32) * np.float32(0.01)


def make_inputs(shape: Shape | tuple, seed: int | None = None, dist: str | None = None):
    """Return (x_bits [M,K], w_bits [N,K], b_bits [N]) as uint16 numpy arrays of bf16.

    ``shape`` is a Shape or an (M, K, N) tuple; ``seed``/``dist`` override the shape's."""
    if isinstance(shape, Shape):
        M, K, N = shape.M, shape.K, shape.N
        seed = shape.seed if seed is None else seed
        dist = shape.dist if dist is None else dist
    else:
        M, K, N = shape
        seed = 12345 if seed is None else seed
        dist = "outlier" if dist is None else dist
    rng = np.random.default_rng(seed)
    x = draw_x(rng, M, K, dist)
    w = draw_w(rng, N, K)
    b = draw_b(rng, N)
    return bf16_bits_from_f32(x), bf16_bits_from_f32(w), bf16_bits_from_f32(b)
