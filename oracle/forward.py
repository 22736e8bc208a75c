"""Bidirectional transformer forward, ``Forward(p_theta, x)`` of Algorithm 1 (Appendix A).

Masked diffusion LMs attend over all positions with no causal mask (Section 1;
Appendix B.2 on LLaDA / Dream). One sequence at a time, float64 throughout.

bf16-boundary mode (default) rounds to bfloat16 exactly where the GPU stores a
bfloat16 tensor, so both sides see the same operands:
  u  = bf16(rmsnorm(r) * g1)                     (attention input)
  q, k, v = bf16(rope(u Wq^T + bq)), ..., bf16(u Wv^T + bv)
  o  = bf16(softmax(q k^T / sqrt(dh)) v)          (per head, all keys)
  r += o Wo^T
  u2 = bf16(rmsnorm(r) * g2)
  a  = bf16(silu(u2 Wg^T) * (u2 Wu^T))
  r += a Wd^T
  h_f = bf16(rmsnorm(r) * gf)
Pure mode (``bf16_boundary=False``) drops those roundings (weights stay as given).
The residual stream r is never rounded.

``dtype=np.float32`` evaluates the same definition in float32 arithmetic. It is not the
reference; it measures how far any float32 implementation of this rounding list lands from the
float64 result, which sizes the whole-step tolerance of the GPU parity tests.

The stage functions (``norm_stage``, ``qkv_stage``, ``attention_stage``, ``swiglu_stage``,
``residual_stage``) are the steps of one layer in the order above; ``forward`` composes them, and the
stage-wise parity tests call them one at a time on given stage inputs.
"""
from typing import Callable, Mapping, Optional, Tuple

import numpy as np

from .numerics import apply_rope, bf16_round, rmsnorm, rope_tables, silu


def _w(weights, name, dtype=np.float64) -> Optional[np.ndarray]:
    v = weights[name] if not callable(weights) else weights(name)
    return None if v is None else np.asarray(v, dtype=dtype)


def norm_stage(r, gain, eps, rnd):
    """u = bf16(rmsnorm(r) * g): the normalised operand of the next projection."""
    return rnd(rmsnorm(r, gain, eps))


def qkv_stage(geom, W, l, u, cos, sin, rnd, rope=True):
    """q, k, v of layer ``l`` for the rows of ``u`` [S, d]: projections (+ bias), rotate-half RoPE on
    q and k at the positions of ``cos``/``sin`` [S, dh/2], then the bf16 storage point.
    Returns q [H, S, dh], k [Hkv, S, dh], v [Hkv, S, dh]."""
    H, Hkv, dh = geom.n_heads, geom.n_kv_heads, geom.head_dim
    S = u.shape[0]
    p = f"l{l}."
    q = u @ W(p + "wq").T
    k = u @ W(p + "wk").T
    v = u @ W(p + "wv").T
    if geom.qkv_bias:
        q = q + W(p + "bq")
        k = k + W(p + "bk")
        v = v + W(p + "bv")
    q = q.reshape(S, H, dh).transpose(1, 0, 2)
    k = k.reshape(S, Hkv, dh).transpose(1, 0, 2)
    v = v.reshape(S, Hkv, dh).transpose(1, 0, 2)
    if rope:
        q = apply_rope(q, cos, sin)
        k = apply_rope(k, cos, sin)
    return rnd(q), rnd(k), rnd(v)


def attention_stage(geom, q, k, v, rnd, dtype=np.float64):
    """o = bf16(softmax(q k^T / sqrt(dh)) v) per head over ALL keys (no mask), query head h reading
    key/value head h // (H / Hkv). q [H, Sq, dh], k and v [Hkv, Sk, dh]; returns o [Sq, H*dh]."""
    H, Hkv, dh = geom.n_heads, geom.n_kv_heads, geom.head_dim
    group = H // Hkv
    Sq = q.shape[1]
    o = np.empty((H, Sq, dh), np.dtype(dtype))
    for h in range(H):
        g = h // group
        s = (q[h] @ k[g].T) / float(np.sqrt(dh))
        s = np.exp(s - s.max(axis=1, keepdims=True))
        P = s / s.sum(axis=1, keepdims=True)
        o[h] = P @ v[g]
    return rnd(o.transpose(1, 0, 2).reshape(Sq, H * dh))


def swiglu_stage(W, l, u2, rnd):
    """a = bf16(silu(u2 Wg^T) * (u2 Wu^T))."""
    p = f"l{l}."
    return rnd(silu(u2 @ W(p + "wg").T) * (u2 @ W(p + "wu").T))


def residual_stage(r, x, w):
    """r + x w^T (the residual stream is never rounded)."""
    return r + x @ w.T


def rounding(bf16_boundary, dtype=np.float64):
    """The storage-point rounding of the chosen mode: bf16 (then widened to ``dtype``) or none."""
    dt = np.dtype(dtype)
    if bf16_boundary:
        return lambda a: bf16_round(a).astype(dt)
    return lambda a: a


def forward(geom, weights, tokens: np.ndarray, positions: np.ndarray,
            kv: Optional[Callable[[int], Tuple[np.ndarray, np.ndarray]]] = None,
            bf16_boundary: bool = True, rope: bool = True, return_residuals: bool = False,
            return_kv: bool = False, dtype=np.float64):
    """Final hidden states h_f [S, d] (float64) of one sequence.

    geom: object with the geometry fields of ``synth.Geometry``.
    weights: mapping or callable name -> array (the float values of the weights).
    tokens: [S] ids; positions: [S] absolute positions used by RoPE.
    kv: optional callable layer -> (Kc [Hkv, P, dh], Vc [Hkv, dh, P]) cached prefix
        (keys already rotated); the S fresh tokens then attend to [cache || fresh].
    rope: False disables the rotary embedding (used by the permutation pin).
    return_residuals: also return the residual stream before layer 0 and after every layer.
    return_kv: also return the per-layer (k [Hkv,S,dh], v [Hkv,dh,S]) of the S tokens, as a cache would
        hold them.
    """
    dt = np.dtype(dtype)
    rnd = rounding(bf16_boundary, dt)
    cos, sin = (t.astype(dt) for t in rope_tables(positions, geom.head_dim, geom.rope_base))
    W = lambda name: _w(weights, name, dt)

    r = W("embed")[np.asarray(tokens)]                           # [S, d]
    residuals = [r.copy()] if return_residuals else None
    kv_out = [] if return_kv else None
    for l in range(geom.n_layers):
        p = f"l{l}."
        u = norm_stage(r, W(p + "g1"), geom.rms_eps, rnd)
        q, k, v = qkv_stage(geom, W, l, u, cos, sin, rnd, rope)
        if return_kv:
            kv_out.append((k.copy(), v.transpose(0, 2, 1).copy()))
        if kv is not None:
            kc, vc = kv(l)
            k = np.concatenate([np.asarray(kc, dt), k], axis=1)
            v = np.concatenate([np.asarray(vc, dt).transpose(0, 2, 1), v], axis=1)
        o = attention_stage(geom, q, k, v, rnd, dt)
        r = residual_stage(r, o, W(p + "wo"))
        u2 = norm_stage(r, W(p + "g2"), geom.rms_eps, rnd)
        a = swiglu_stage(W, l, u2, rnd)
        r = residual_stage(r, a, W(p + "wd"))
        if return_residuals:
            residuals.append(r.copy())
    hf = norm_stage(r, W("gf"), geom.rms_eps, rnd)
    extra = ([residuals] if return_residuals else []) + ([kv_out] if return_kv else [])
    return (hf, *extra) if extra else hf


def lm_logits(weights, hf: np.ndarray, chunk: int = 8192, dtype=np.float64) -> np.ndarray:
    """logits = h_f W_lm^T in float64 (or ``dtype``), never rounded; [R, V]. Vocabulary in chunks."""
    from .numerics import WeightView, weight_values
    if isinstance(weights, WeightView):
        raw = weights.stored["lm_head"]
        get = lambda a, b: weight_values(raw[a:b], weights.bf16_boundary).astype(dtype)
        V = raw.shape[0]
    else:
        W = weights["lm_head"] if not callable(weights) else weights("lm_head")
        get = lambda a, b: np.asarray(W[a:b], dtype)
        V = W.shape[0]
    out = np.empty((hf.shape[0], V), dtype)
    hf = np.asarray(hf, dtype)
    for v0 in range(0, V, chunk):
        out[:, v0:v0 + chunk] = hf @ get(v0, v0 + chunk).T
    return out
