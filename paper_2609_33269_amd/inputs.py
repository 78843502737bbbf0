"""Seeded synthetic inputs for the ASP linear layer.

This module only draws random numbers and shapes them into the workloads the
layer is measured on.  It holds none of the layer's own arithmetic: no
smoothing factor, no eigen-decomposition, no quantizer, no packing.  Both the
CPU oracle (through the tests) and the GPU path consume exactly the arrays it
returns, so a mismatch between the two can never come from here.

Conventions
-----------
* ``x``: activations, bf16 bit patterns, shape ``[M][K]`` (row = token).
* ``w``: weight, bf16 bit patterns, shape ``[N][K]`` (row = output channel),
  i.e. the transpose of the paper's ``W in R^{d x d'}`` (Sec. 3, "Post-Training
  Quantization": ``y = W^T x``).
* ``a``: float64 ``[K][64]`` factor of the stand-in Gramian
  ``G = A A^T / K + 1e-3 I`` that replaces the Action Observability Gramian
  (Sec. 4.1, Eq. 5), which needs a trained model to estimate.
* ``bias``: optional bf16 ``[N]``.

All draws come from numpy's PCG64 seeded with ``(seed, stream...)`` tuples, in
a fixed order, so every array is reproducible on any host.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np

GRAM_COLS = 64          # columns of the Gramian factor A (rank of the stand-in AOG)
GROUP = 64              # quantization group along K


def f32_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return uint16 bits.

    Used to make the synthetic tensors bf16-valued, as the workloads are.
    """
    u = np.ascontiguousarray(v, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class LayerShape:
    """One ASP linear: ``M`` tokens, ``K`` inputs, ``N`` outputs, rank ``r``."""
    M: int
    K: int
    N: int
    r: int
    name: str = ""


@dataclass
class ActRecipe:
    """How the activation tensor is drawn.

    kind = "outlier": N(0,1) with a fraction (or a fixed count) of channels
    multiplied by a factor, either fixed or log-uniform in [lo, hi].
    kind = "gelu": bf16 of the exact-erf GELU of N(0,1) (the input of an FFN
    down-projection, heavy positive tail).
    """
    kind: str = "outlier"
    n_outliers: Optional[int] = None
    frac_outliers: float = 0.0
    factor: Optional[float] = 20.0
    log_uniform: Tuple[float, float] = (10.0, 50.0)


@dataclass
class WeightRecipe:
    """Weight entries N(0, std^2); ``std=None`` means std = 1/sqrt(K)."""
    std: Optional[float] = None


@dataclass
class LayerDraws:
    shape: LayerShape
    x: np.ndarray                 # uint16 [M][K] bf16 bits
    w: np.ndarray                 # uint16 [N][K] bf16 bits
    a: np.ndarray                 # float64 [K][64]
    outlier_channels: np.ndarray  # int64 indices
    bias: Optional[np.ndarray] = None   # uint16 [N] bf16 bits
    seed: tuple = field(default_factory=tuple)


def _rng(*seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(list(seed)))


def _gelu_erf(z: np.ndarray) -> np.ndarray:
    from scipy.special import erf
    z64 = z.astype(np.float64)
    return (0.5 * z64 * (1.0 + erf(z64 / np.sqrt(2.0)))).astype(np.float32)


def draw_activations(M: int, K: int, recipe: ActRecipe, rng: np.random.Generator):
    """Draw ``x`` (bf16 bits, [M][K]) and the indices of its outlier channels."""
    z = rng.standard_normal((M, K), dtype=np.float32)
    if recipe.kind == "gelu":
        return f32_to_bf16_bits(_gelu_erf(z)), np.zeros(0, dtype=np.int64)
    if recipe.n_outliers is not None:
        n_out = int(recipe.n_outliers)
    else:
        n_out = int(round(recipe.frac_outliers * K))
    n_out = min(max(n_out, 0), K)
    ch = np.sort(rng.choice(K, size=n_out, replace=False)).astype(np.int64)
    if recipe.factor is not None:
        fac = np.full(n_out, recipe.factor, dtype=np.float32)
    else:
        lo, hi = recipe.log_uniform
        fac = np.exp(rng.uniform(np.log(lo), np.log(hi), size=n_out)).astype(np.float32)
    if n_out:
        z[:, ch] *= fac[None, :]
    return f32_to_bf16_bits(z), ch


def draw_layer(shape: LayerShape, act: ActRecipe, wrec: WeightRecipe, seed: tuple,
               with_bias: bool = False) -> LayerDraws:
    """Draw one layer's tensors in a fixed order: x, outliers, W, A, bias."""
    rng = _rng(*seed)
    x, ch = draw_activations(shape.M, shape.K, act, rng)
    std = (1.0 / np.sqrt(shape.K)) if wrec.std is None else wrec.std
    w = f32_to_bf16_bits(rng.standard_normal((shape.N, shape.K), dtype=np.float32) * np.float32(std))
    a = rng.standard_normal((shape.K, GRAM_COLS))
    bias = None
    if with_bias:
        bias = f32_to_bf16_bits(rng.standard_normal(shape.N, dtype=np.float32) * np.float32(0.02))
    return LayerDraws(shape=shape, x=x, w=w, a=a, outlier_channels=ch, bias=bias, seed=tuple(seed))


# ---------------------------------------------------------------------------
# The named workloads.  Each returns LayerDraws (or a list of them).
# ---------------------------------------------------------------------------

def tiny(seed: int = 0, with_bias: bool = False) -> LayerDraws:
    """64 tokens, 256 -> 256, rank 16; 4 outlier channels x20; W ~ N(0, 0.02^2)."""
    return draw_layer(LayerShape(64, 256, 256, 16, "tiny"),
                      ActRecipe(n_outliers=4, factor=20.0), WeightRecipe(std=0.02),
                      (seed, 0), with_bias)


def video_dit_qkv(seed: int = 1, M: int = 4096) -> LayerDraws:
    """Attention QKV projection: 4096 tokens, 3072 -> 9216, rank 32; 1% of
    channels scaled by a log-uniform factor in [10, 50]; W ~ N(0, 1/K)."""
    return draw_layer(LayerShape(M, 3072, 9216, 32, "video_dit_qkv"),
                      ActRecipe(frac_outliers=0.01, factor=None), WeightRecipe(),
                      (seed, 0))


def video_dit_ffn_up(seed: int = 2, M: int = 4096) -> LayerDraws:
    """FFN up-projection: 4096 tokens, 3072 -> 14336, rank 32 (activations as QKV)."""
    return draw_layer(LayerShape(M, 3072, 14336, 32, "video_dit_ffn_up"),
                      ActRecipe(frac_outliers=0.01, factor=None), WeightRecipe(),
                      (seed, 0))


def video_dit_ffn_down(seed: int = 2, M: int = 4096) -> LayerDraws:
    """FFN down-projection: 4096 tokens, 14336 -> 3072, rank 32; input = GELU(N(0,1))."""
    return draw_layer(LayerShape(M, 14336, 3072, 32, "video_dit_ffn_down"),
                      ActRecipe(kind="gelu"), WeightRecipe(), (seed, 1))


ACTION_EXPERT_SHAPES = [(M, N) for M in (16, 32, 64) for N in (4096, 1024)]


def action_expert(M: int, N: int, seed: int = 3) -> LayerDraws:
    """Small-M action-expert linear: M in {16,32,64}, 1024 -> N in {4096,1024},
    rank 16; 2% of channels x20; W ~ N(0, 1/K).  One sub-seed per shape."""
    idx = ACTION_EXPERT_SHAPES.index((M, N)) if (M, N) in ACTION_EXPERT_SHAPES else 100 + M * 7 + N
    return draw_layer(LayerShape(M, 1024, N, 16, f"action_expert_m{M}_n{N}"),
                      ActRecipe(frac_outliers=0.02, factor=20.0), WeightRecipe(),
                      (seed, idx))


DENOISE_BLOCK = [("qkv", 3072, 9216), ("out", 3072, 3072), ("ffn_up", 3072, 14336),
                 ("ffn_down", 14336, 3072)]
DENOISE_BLOCKS = 30


def denoise_step_layer(block: int, which: int, seed: int = 4, M: int = 8192) -> LayerDraws:
    """One layer of a 30-block denoising step (hidden 3072, FFN 14336, 8192 tokens).

    Each layer has its own seeded weights and a fresh seeded activation with 1%
    log-uniform outlier channels (the down-projection gets a GELU input).
    """
    name, K, N = DENOISE_BLOCK[which]
    act = ActRecipe(kind="gelu") if name == "ffn_down" else ActRecipe(frac_outliers=0.01, factor=None)
    return draw_layer(LayerShape(M, K, N, 32, f"denoise_b{block}_{name}"), act, WeightRecipe(),
                      (seed, block, which))


def custom(M: int, K: int, N: int, r: int, seed: int, n_outliers: int = 0,
           factor: float = 20.0, wstd: Optional[float] = None, with_bias: bool = False) -> LayerDraws:
    """Arbitrary shape for edge-case tests (ragged M, K = 64, ...)."""
    return draw_layer(LayerShape(M, K, N, r, f"custom_{M}x{K}x{N}_r{r}"),
                      ActRecipe(n_outliers=n_outliers, factor=factor), WeightRecipe(std=wstd),
                      (seed, 7), with_bias)
