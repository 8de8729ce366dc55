"""Seeded synthetic inputs for FFF layers.

This module only draws random numbers and changes their storage type; it
holds none of the FFF arithmetic.  Both the HIP path and the fp64 oracle are
fed from it, so it is the one piece of code they share.

Recipe (the paper publishes no weights we can use here, and its speed
benchmark is shape-only: 128 sequences of 128 tokens, hidden width 768,
Section 3.3):

* every tensor comes from ``numpy.random.default_rng([seed, layer, tensor])``
  with tensor 0 = x, 1 = W_in, 2 = W_out, 3 = LayerNorm gain, 4 = LayerNorm
  shift;
* x ~ N(0, 1), drawn as float32;
* W_in, W_out ~ N(0, 1/H) (variance 1/H, so logits are roughly N(0, 1)),
  drawn as float32 and multiplied by float32(1/sqrt(H));
* LayerNorm gain 1 + 0.1 N(0, 1) and shift 0.1 N(0, 1), float32 (trained
  values are not available; these keep the normalised input near unit scale);
* bf16 tensors are the round-to-nearest-even bf16 of those float32 draws,
  stored as their uint16 bit patterns.

Layouts: x is [B, H] row-major; W_in and W_out are [T, N, H] with
N = 2**(D+1) - 1 nodes per tree in heap order.
"""
from __future__ import annotations

import numpy as np

F32 = "f32"
BF16 = "bf16"
DTYPES = (F32, BF16)

TENSOR_X, TENSOR_W_IN, TENSOR_W_OUT, TENSOR_GAMMA, TENSOR_BETA = 0, 1, 2, 3, 4


def n_nodes(depth: int) -> int:
    """Nodes in one balanced tree with ``depth`` edges on a root-to-leaf path."""
    return (1 << (depth + 1)) - 1


def gaussian_f32(seed_words, shape, scale: float | None = None) -> np.ndarray:
    """float32 standard normal draw from a seed sequence, optionally scaled in float32."""
    rng = np.random.default_rng(list(seed_words))
    a = rng.standard_normal(size=shape, dtype=np.float32)
    if scale is not None:
        a *= np.float32(scale)
    return a


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns uint16 bit patterns.

    NaNs map to a quiet NaN; infinities are kept.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        rounded[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return rounded


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32)


def as_dtype(a_f32: np.ndarray, dtype: str) -> np.ndarray:
    """Store a float32 draw as ``dtype``: float32 itself, or bf16 bit patterns."""
    if dtype == F32:
        return np.ascontiguousarray(a_f32, dtype=np.float32)
    if dtype == BF16:
        return f32_to_bf16_bits(a_f32)
    raise ValueError(f"unknown dtype {dtype!r}")


def make_x(seed: int, n_tokens: int, hidden: int, x_dtype: str, layer: int = 0) -> np.ndarray:
    return as_dtype(gaussian_f32((seed, layer, TENSOR_X), (n_tokens, hidden)), x_dtype)


def make_weights(seed: int, hidden: int, depth: int, n_trees: int, w_dtype: str,
                 layer: int = 0) -> tuple[np.ndarray, np.ndarray]:
    shape = (n_trees, n_nodes(depth), hidden)
    scale = 1.0 / np.sqrt(np.float64(hidden))
    w_in = gaussian_f32((seed, layer, TENSOR_W_IN), shape, scale)
    w_out = gaussian_f32((seed, layer, TENSOR_W_OUT), shape, scale)
    return as_dtype(w_in, w_dtype), as_dtype(w_out, w_dtype)


def make_norm(seed: int, hidden: int, layer: int = 0) -> tuple[np.ndarray, np.ndarray]:
    """float32 LayerNorm gain and shift of one layer."""
    gamma = np.float32(1.0) + gaussian_f32((seed, layer, TENSOR_GAMMA), (hidden,), 0.1)
    beta = gaussian_f32((seed, layer, TENSOR_BETA), (hidden,), 0.1)
    return gamma.astype(np.float32), beta


def make_layer(seed: int, n_tokens: int, hidden: int, depth: int, n_trees: int,
               x_dtype: str, w_dtype: str, layer: int = 0) -> dict:
    """x, W_in, W_out for one FFF layer, stored in the requested dtypes."""
    x = make_x(seed, n_tokens, hidden, x_dtype, layer)
    w_in, w_out = make_weights(seed, hidden, depth, n_trees, w_dtype, layer)
    return {"x": x, "w_in": w_in, "w_out": w_out}


def make_clustered_x(seed: int, n_tokens: int, hidden: int, x_dtype: str, n_centres: int = 64,
                     spread: float = 0.1, layer: int = 0) -> np.ndarray:
    """Skewed-routing stress input: x_b = c_j(b) + spread * eps, with ``n_centres`` centres.

    Tokens near one centre tend to share tree paths, so bucket sizes become uneven.
    """
    rng = np.random.default_rng([seed, layer, TENSOR_X, 1])
    centres = rng.standard_normal(size=(n_centres, hidden), dtype=np.float32)
    which = rng.integers(0, n_centres, size=n_tokens)
    eps = rng.standard_normal(size=(n_tokens, hidden), dtype=np.float32)
    x = centres[which] + np.float32(spread) * eps
    return as_dtype(x, x_dtype)


def small_int_layer(seed: int, n_tokens: int, hidden: int, depth: int, n_trees: int,
                    lo: int = -3, hi: int = 3) -> dict:
    """Small-integer x and weights (float32 storage): every product and partial sum is exact."""
    rng = np.random.default_rng([seed, 99])
    N = n_nodes(depth)
    x = rng.integers(lo, hi + 1, size=(n_tokens, hidden)).astype(np.float32)
    w_in = rng.integers(lo, hi + 1, size=(n_trees, N, hidden)).astype(np.float32)
    w_out = rng.integers(lo, hi + 1, size=(n_trees, N, hidden)).astype(np.float32)
    return {"x": x, "w_in": w_in, "w_out": w_out}
