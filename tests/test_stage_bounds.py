"""CPU pins of the stage-wise checks (stage_checks.py) that the full-size GPU parity tests use.

Two properties make the checks meaningful:
* a float32 implementation of each stage passes them: the oracle's own stage functions evaluated in
  float32 arithmetic (numpy's float32 BLAS, another summation order than the GPU's) stay inside every
  derived bound, on a Dream-style geometry (GQA, q/k/v biases, head_dim 128) with a cached prefix;
* plausible mistakes fail them: a bias added after the rotation, keys rotated at positions shifted by
  one, a dropped residual term, a transposed operand.
"""
import dataclasses

import numpy as np
import pytest

import synth
from oracle.forward import attention_stage, norm_stage, qkv_stage, residual_stage, swiglu_stage
from oracle.numerics import WeightView, bf16_round, rope_tables

import stage_checks as sc

GEOM = dataclasses.replace(synth.WORKLOADS["c1s"].geom, name="stage-pin", n_layers=1, n_heads=4, n_kv_heads=2,
                           head_dim=128, d_model=384, d_ffn=768, qkv_bias=True, weight_dtype="bf16",
                           rope_base=1e6, rms_eps=1e-6)
ident = lambda a: a


def _bits(x):
    return (bf16_round(np.asarray(x, np.float64)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


@pytest.fixture(scope="module")
def setup():
    stored = synth.make_weights(GEOM)
    W64 = WeightView(stored)
    W = {k: W64(k) for k in stored if stored[k] is not None}
    W32 = {k: v.astype(np.float32) for k, v in W.items()}
    rng = np.random.default_rng(3)
    S, P = 40, 24
    r = (rng.standard_normal((S, GEOM.d_model)) * 2).astype(np.float32).astype(np.float64)
    kc = bf16_round(rng.standard_normal((GEOM.n_kv_heads, P, GEOM.head_dim)))
    vc = bf16_round(rng.standard_normal((GEOM.n_kv_heads, P, GEOM.head_dim)))
    cos, sin = rope_tables(P + np.arange(S), GEOM.head_dim, GEOM.rope_base)
    return W, W32, r, kc, vc, cos, sin


def _float32_stages(W32, r, kc, vc, cos, sin):
    """The layer's stages in float32 arithmetic, each fed the previous float32 stage's bf16 output."""
    g = GEOM
    rnd32 = lambda a: bf16_round(a).astype(np.float32)
    f = lambda n: W32[n]
    out = {}
    r32 = r.astype(np.float32)
    out["u"] = norm_stage(r32, f("l0.g1"), g.rms_eps, ident)
    u = rnd32(out["u"])
    q, k, v = qkv_stage(g, f, 0, u, cos.astype(np.float32), sin.astype(np.float32), ident)
    out["q"], out["k"], out["v"] = q, k, v
    q, k, v = rnd32(q), rnd32(k), rnd32(v)
    kk = np.concatenate([kc.astype(np.float32), k], axis=1)
    vv = np.concatenate([vc.astype(np.float32), v], axis=1)
    out["o"] = attention_stage(g, q, kk, vv, ident, np.float32)
    o = rnd32(out["o"])
    out["r_mid"] = residual_stage(r32, o, f("l0.wo"))
    out["u2"] = norm_stage(out["r_mid"], f("l0.g2"), g.rms_eps, ident)
    u2 = rnd32(out["u2"])
    out["a"] = swiglu_stage(f, 0, u2, ident)
    a = rnd32(out["a"])
    out["r_out"] = residual_stage(out["r_mid"], a, f("l0.wd"))
    return out, dict(u=u, q=q, k=k, v=v, o=o, u2=u2, a=a)


def _check_all(W, r, kc, vc, cos, sin, got, inputs, wrong=None):
    """Exact stage values on the float32 side's inputs, then every check. `wrong` plants a mistake."""
    g = GEOM
    H, Hkv, dh, d = g.n_heads, g.n_kv_heads, g.head_dim, g.d_model
    f = lambda n: W[n]
    rep = {}
    x = norm_stage(r, f("l0.g1"), g.rms_eps, ident)
    sc.check_bf16("u", _bits(got["u"]), x, sc.norm_bound(x, d), rep)
    u = inputs["u"].astype(np.float64)
    c_, s_ = (cos, sin) if wrong != "rope_shift" else rope_tables(25 + np.arange(len(r)), dh, g.rope_base)
    qx, kx, vx = qkv_stage(g, f, 0, u, c_, s_, ident)
    if wrong == "bias_after_rope":
        b = lambda n, h: f("l0." + n).reshape(h, 1, dh)
        qx = qkv_stage(dataclasses.replace(g, qkv_bias=False), f, 0, u, c_, s_, ident)[0] + b("bq", H)
    pre = {}
    for nm, heads, wn, bn in (("q", H, "wq", "bq"), ("k", Hkv, "wk", "bk"), ("v", Hkv, "wv", "bv")):
        E = sc.linear_bound(np.abs(u), np.abs(f("l0." + wn)), np.abs(f("l0." + bn)))
        val = u @ f("l0." + wn).T + f("l0." + bn)
        pre[nm] = (E.reshape(-1, heads, dh).transpose(1, 0, 2), val.reshape(-1, heads, dh).transpose(1, 0, 2))
    sc.check_bf16("q", _bits(got["q"]), qx, sc.rope_pair_bound(*pre["q"], dh // 2), rep)
    sc.check_bf16("k", _bits(got["k"]), kx, sc.rope_pair_bound(*pre["k"], dh // 2), rep)
    sc.check_bf16("v", _bits(got["v"]), vx, pre["v"][0], rep)
    q, k, v = (inputs[n].astype(np.float64) for n in ("q", "k", "v"))
    kk, vv = np.concatenate([kc, k], axis=1), np.concatenate([vc, v], axis=1)
    if wrong == "transposed_v":
        vv = vv[:, ::-1]
    ex = attention_stage(g, q, kk, vv, ident)
    E = np.empty_like(ex)
    for h in range(H):
        s = q[h] @ kk[h // 2].T / np.sqrt(dh)
        Pm = np.exp(s - s.max(1, keepdims=True))
        Pm /= Pm.sum(1, keepdims=True)
        E[:, h * dh:(h + 1) * dh] = sc.attention_bound(q[h], kk[h // 2], vv[h // 2], Pm, np.log2(np.e) / np.sqrt(dh))
    sc.check_bf16("o", _bits(got["o"]), ex, E, rep)
    o = inputs["o"].astype(np.float64)
    base = r if wrong != "dropped_residual" else 0 * r
    sc.check_f32("r_mid", got["r_mid"], residual_stage(base, o, f("l0.wo")),
                 sc.linear_bound(np.abs(o), np.abs(f("l0.wo")), np.abs(r), extra_terms=4), rep)
    rm = got["r_mid"].astype(np.float64)
    x2 = norm_stage(rm, f("l0.g2"), g.rms_eps, ident)
    sc.check_bf16("u2", _bits(got["u2"]), x2, sc.norm_bound(x2, d), rep)
    u2 = inputs["u2"].astype(np.float64)
    gate, up = u2 @ f("l0.wg").T, u2 @ f("l0.wu").T
    Eg = sc.linear_bound(np.abs(u2), np.abs(f("l0.wg")))
    Eu = sc.linear_bound(np.abs(u2), np.abs(f("l0.wu")))
    sc.check_bf16("a", _bits(got["a"]), swiglu_stage(f, 0, u2, ident), sc.swiglu_bound(gate, up, Eg, Eu), rep)
    a = inputs["a"].astype(np.float64)
    sc.check_f32("r_out", got["r_out"], residual_stage(rm, a, f("l0.wd")),
                 sc.linear_bound(np.abs(a), np.abs(f("l0.wd")), np.abs(rm), extra_terms=4), rep)
    return rep


def test_float32_evaluation_meets_every_stage_bound(setup):
    W, W32, r, kc, vc, cos, sin = setup
    got, inputs = _float32_stages(W32, r, kc, vc, cos, sin)
    rep = _check_all(W, r, kc, vc, cos, sin, got, inputs)
    print(rep)
    # the bounds are not vacuous: the float32 residual errors are a small but visible part of them
    assert 0 < rep["r_out"]["max_ratio_to_bound"] < 1
    assert all(v["flip_fraction"] < 0.01 for v in rep.values() if "flip_fraction" in v)


@pytest.mark.parametrize("wrong", ["bias_after_rope", "rope_shift", "transposed_v", "dropped_residual"])
def test_planted_mistakes_fail_the_checks(setup, wrong):
    W, W32, r, kc, vc, cos, sin = setup
    got, inputs = _float32_stages(W32, r, kc, vc, cos, sin)
    with pytest.raises(AssertionError):
        _check_all(W, r, kc, vc, cos, sin, got, inputs, wrong=wrong)


def test_bf16_check_accepts_one_sided_flips_only_inside_the_bound():
    exact = np.array([1.0 + 2.0 ** -8 + 1e-9, 1.0 + 2.0 ** -8 - 1e-9, 1.5, 1.5])
    # a midpoint-adjacent value may round either way when the bound reaches the midpoint ...
    sc.check_bf16("x", _bits([1.0, 1.0 + 2.0 ** -7, 1.5, 1.5]), exact, np.array([1e-8, 1e-8, 0, 0]), {}, max_flip=1)
    # ... but not when the bound is smaller than the distance to the midpoint
    with pytest.raises(AssertionError):
        sc.check_bf16("x", _bits([1.0, 1.0, 1.5, 1.5]), exact, np.array([1e-10, 1e-10, 0, 0]), {}, max_flip=1)
    # and never by two ulps when the bound is below half an ulp
    with pytest.raises(AssertionError):
        sc.check_bf16("x", _bits([1.0 + 2.0 ** -6, 1.0, 1.5, 1.5]), exact, np.array([1e-4, 1e-8, 0, 0]), {},
                      max_flip=1)
    # too many flips
    with pytest.raises(AssertionError):
        sc.check_bf16("x", _bits([1.0, 1.0 + 2.0 ** -7, 1.5, 1.5]), exact, np.array([1e-8, 1e-8, 0, 0]), {})
