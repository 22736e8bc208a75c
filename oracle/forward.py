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
"""
from typing import Callable, Mapping, Optional, Tuple

import numpy as np

from .numerics import apply_rope, bf16_round, rmsnorm, rope_tables, silu


def _w(weights, name, dtype=np.float64) -> Optional[np.ndarray]:
    v = weights[name] if not callable(weights) else weights(name)
    return None if v is None else np.asarray(v, dtype=dtype)


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
    return_kv: also return the per-layer (k [Hkv,S,dh], v [Hkv,dh,S]) of the S tokens, as a cache would
        hold them.
    """
    dt = np.dtype(dtype)
    if bf16_boundary:
        rnd = lambda a: bf16_round(a).astype(dt)
    else:
        rnd = lambda a: a
    d, H, Hkv, dh = geom.d_model, geom.n_heads, geom.n_kv_heads, geom.head_dim
    S = len(tokens)
    group = H // Hkv
    cos, sin = (t.astype(dt) for t in rope_tables(positions, dh, geom.rope_base))
    W = lambda name: _w(weights, name, dt)

    r = W("embed")[np.asarray(tokens)]                           # [S, d]
    residuals = [r.copy()] if return_residuals else None
    kv_out = [] if return_kv else None
    for l in range(geom.n_layers):
        p = f"l{l}."
        u = rnd(rmsnorm(r, W(p + "g1"), geom.rms_eps))
        q = u @ W(p + "wq").T
        k = u @ W(p + "wk").T
        v = u @ W(p + "wv").T
        if geom.qkv_bias:
            q = q + W(p + "bq")
            k = k + W(p + "bk")
            v = v + W(p + "bv")
        q = q.reshape(S, H, dh).transpose(1, 0, 2)                # [H, S, dh]
        k = k.reshape(S, Hkv, dh).transpose(1, 0, 2)              # [Hkv, S, dh]
        v = v.reshape(S, Hkv, dh).transpose(1, 0, 2)
        if rope:
            q = apply_rope(q, cos, sin)
            k = apply_rope(k, cos, sin)
        q, k, v = rnd(q), rnd(k), rnd(v)
        if return_kv:
            kv_out.append((k.copy(), v.transpose(0, 2, 1).copy()))
        if kv is not None:
            kc, vc = kv(l)
            k = np.concatenate([np.asarray(kc, dt), k], axis=1)
            v = np.concatenate([np.asarray(vc, dt).transpose(0, 2, 1), v], axis=1)
        o = np.empty((H, S, dh), dt)
        for h in range(H):
            g = h // group
            s = (q[h] @ k[g].T) / float(np.sqrt(dh))                     # [S, Sk], no mask
            s = np.exp(s - s.max(axis=1, keepdims=True))
            P = s / s.sum(axis=1, keepdims=True)
            o[h] = P @ v[g]
        o = rnd(o.transpose(1, 0, 2).reshape(S, H * dh))
        r = r + o @ W(p + "wo").T
        u2 = rnd(rmsnorm(r, W(p + "g2"), geom.rms_eps))
        a = rnd(silu(u2 @ W(p + "wg").T) * (u2 @ W(p + "wu").T))
        r = r + a @ W(p + "wd").T
        if return_residuals:
            residuals.append(r.copy())
    hf = rnd(rmsnorm(r, W("gf"), geom.rms_eps))
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
