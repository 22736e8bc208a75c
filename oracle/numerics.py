"""Elementwise numerics of the LLaMA-style mask predictor, float64.

The paper does not describe the architecture; its base models (LLaDA-8B,
LLaDA-1.5, Dream-7B, Section 4 setup) are pre-norm transformers with RMSNorm,
rotary position embeddings (rotate-half form) and SwiGLU feed-forward blocks.
"""
import numpy as np


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value, ties to even; returns float64.

    bfloat16 keeps 8 significant bits. Writing x = m * 2**e with 0.5 <= |m| < 1,
    the rounded value is rint(m * 2**8) * 2**(e - 8); numpy's rint rounds half
    to even. Direct rounding from float64 (no float32 step). Values below the
    bfloat16 normal range are rounded on the same 8-bit grid (no subnormal
    flush); activations here are far from that range.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def rmsnorm(r: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """r / sqrt(mean(r^2) + eps) * gain over the last axis.

    Evaluated in float32 when ``r`` is float32 (the float32 evaluation of the whole definition,
    used only to size tolerances), in float64 otherwise."""
    r = np.asarray(r)
    dt = np.float32 if r.dtype == np.float32 else np.float64
    r = r.astype(dt, copy=False)
    ms = np.mean(r * r, axis=-1, keepdims=True, dtype=dt)
    inv = dt(1.0) / np.sqrt(ms + dt(eps))
    return (r * inv) * np.asarray(gain, dtype=dt)


def rope_tables(positions: np.ndarray, head_dim: int, base: float):
    """cos/sin of theta_{pos,i} = pos * base^(-2i/head_dim), i < head_dim/2; shapes [S, head_dim/2]."""
    half = head_dim // 2
    inv_freq = base ** (-(2.0 * np.arange(half, dtype=np.float64)) / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half RoPE on x [..., S, head_dim] with tables [S, head_dim/2].

    Pairs (i, i + head_dim/2): (a, b) -> (a cos - b sin, b cos + a sin).
    """
    half = x.shape[-1] // 2
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * cos - b * sin, b * cos + a * sin], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    """x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def weight_values(w: np.ndarray, bf16_boundary: bool = True) -> np.ndarray:
    """Float64 values of a stored weight tensor.

    uint16 arrays are bfloat16 bit patterns (widened exactly). Float arrays are
    rounded to bfloat16 in bf16-boundary mode (the GPU stores every matrix as
    bfloat16) and kept as they are in pure mode.
    """
    w = np.asarray(w)
    if w.dtype == np.uint16:
        return (w.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    w = w.astype(np.float64)
    return bf16_round(w) if bf16_boundary else w


class WeightView:
    """Callable name -> float64 values, converting lazily (one tensor at a time)."""

    def __init__(self, stored, bf16_boundary: bool = True):
        self.stored = stored
        self.bf16_boundary = bf16_boundary

    def __call__(self, name):
        v = self.stored[name]
        return None if v is None else weight_values(v, self.bf16_boundary)

    def __getitem__(self, name):
        return self(name)
