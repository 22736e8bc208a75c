"""Pins for the oracle's elementwise numerics and transformer forward (CPU).

The paper prints no numbers for the forward, so these pins are library routines
(torch.nn.functional in float64, numpy complex arithmetic), textbook identities
and invariants.
"""
import dataclasses

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle.numerics import WeightView, apply_rope, bf16_round, rmsnorm, rope_tables, silu


def test_bf16_round_matches_torch_rne():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000) * 10.0 ** rng.integers(-6, 6, 100000),
                        [0.0, -0.0, 1.0, -2.0, 3.0e38, 1e-30]]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(bf16_round(x.astype(np.float64)), ref)


def test_bf16_round_ties_to_even():
    # 1 + 2^-8 is exactly halfway between 1 and 1 + 2^-7: ties to even -> 1.
    assert bf16_round(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 (odd mantissa) and 1 + 2^-6 (even) -> 1 + 2^-6.
    assert bf16_round(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6
    # just above the tie rounds up; float64 keeps the offset that float32 would lose
    assert bf16_round(np.array([1.0 + 2.0 ** -8 + 2.0 ** -40]))[0] == 1.0 + 2.0 ** -7
    assert bf16_round(np.array([-(1.0 + 2.0 ** -8 + 2.0 ** -40)]))[0] == -(1.0 + 2.0 ** -7)


def test_weight_values_widen_bf16_bits_exactly():
    """Stored weights: bf16 bit patterns widen exactly (as torch's bfloat16 -> float64), float arrays round
    to bf16 in bf16-boundary mode and stay as they are in pure mode."""
    from oracle.numerics import weight_values
    rng = np.random.default_rng(11)
    x = (rng.standard_normal(5000) * 0.05).astype(np.float32)
    bits = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(weight_values(bits), ref)
    np.testing.assert_array_equal(weight_values(x.astype(np.float64)), ref)
    np.testing.assert_array_equal(weight_values(x, bf16_boundary=False), x.astype(np.float64))


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(1)
    r = rng.standard_normal((7, 96)) * 3
    g = rng.standard_normal(96)
    ref = F.rms_norm(torch.from_numpy(r), (96,), torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(rmsnorm(r, g, 1e-5), ref, rtol=1e-13, atol=1e-13)


def test_silu_matches_torch():
    x = np.linspace(-20, 20, 1001)
    np.testing.assert_allclose(silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-13, atol=1e-15)


def test_rope_matches_complex_rotation():
    """Rotate-half RoPE equals multiplying (a_i + i b_i) by exp(i theta_i), theta_i = pos base^(-2i/dh)."""
    rng = np.random.default_rng(2)
    dh, S, base = 64, 37, 1e4
    x = rng.standard_normal((3, S, dh))
    pos = rng.integers(0, 5000, S)
    cos, sin = rope_tables(pos, dh, base)
    got = apply_rope(x, cos, sin)
    z = (x[..., :dh // 2] + 1j * x[..., dh // 2:])
    theta = pos[:, None] * (base ** (-np.arange(0, dh, 2) / dh))[None, :]
    zr = z * np.exp(1j * theta)
    np.testing.assert_allclose(got, np.concatenate([zr.real, zr.imag], -1), rtol=1e-12, atol=1e-12)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(3)
    dh = 128
    q = rng.standard_normal(dh)
    k = rng.standard_normal(dh)
    c0, s0 = rope_tables(np.array([0]), dh, 5e5)
    np.testing.assert_array_equal(apply_rope(q[None], c0, s0)[0], q)          # identity at pos 0
    c, s = rope_tables(np.array([1234]), dh, 5e5)
    np.testing.assert_allclose(np.linalg.norm(apply_rope(q[None], c, s)), np.linalg.norm(q), rtol=1e-13)
    dots = []
    for m in (10, 500, 1200):                                                  # depends on m - n only
        cm, sm = rope_tables(np.array([m]), dh, 5e5)
        cn, sn = rope_tables(np.array([m - 7]), dh, 5e5)
        dots.append(apply_rope(q[None], cm, sm)[0] @ apply_rope(k[None], cn, sn)[0])
    np.testing.assert_allclose(dots, dots[0], rtol=1e-9)


def _torch_forward(geom, W, tokens, positions, bf16_boundary=True, bias_after_rope=False):
    """Second opinion from torch.nn.functional (float64): rms_norm, complex RoPE, SDPA, silu."""
    t = lambda n: torch.from_numpy(np.asarray(W(n), np.float64))
    d, H, Hkv, dh = geom.d_model, geom.n_heads, geom.n_kv_heads, geom.head_dim
    S = len(tokens)
    if bf16_boundary:   # float64 -> float32 -> bfloat16: a second (double-rounding) opinion
        rnd = lambda a: a.to(torch.float32).to(torch.bfloat16).to(torch.float64)
    else:
        rnd = lambda a: a
    theta = torch.from_numpy(np.asarray(positions, np.float64))[:, None] * \
        geom.rope_base ** (-torch.arange(0, dh, 2, dtype=torch.float64) / dh)[None, :]
    rot = torch.polar(torch.ones_like(theta), theta)

    def rope(x):                         # x [h, S, dh]
        z = torch.complex(x[..., :dh // 2], x[..., dh // 2:]) * rot
        return torch.cat([z.real, z.imag], -1)

    r = t("embed")[torch.from_numpy(np.asarray(tokens))]
    for l in range(geom.n_layers):
        p = f"l{l}."
        u = rnd(F.rms_norm(r, (d,), t(p + "g1"), eps=geom.rms_eps))
        # nn.Linear with bias (Qwen2.5 / Dream geometry), before the rotation; bias_after_rope is the
        # plausible mistake the pin must reject
        bias = (lambda n: t(p + n)) if geom.qkv_bias and not bias_after_rope else (lambda n: None)
        q = F.linear(u, t(p + "wq"), bias("bq")).view(S, H, dh).transpose(0, 1)
        k = F.linear(u, t(p + "wk"), bias("bk")).view(S, Hkv, dh).transpose(0, 1)
        v = F.linear(u, t(p + "wv"), bias("bv")).view(S, Hkv, dh).transpose(0, 1)
        q, k = rope(q), rope(k)
        if geom.qkv_bias and bias_after_rope:
            q = q + t(p + "bq").view(H, 1, dh)
            k = k + t(p + "bk").view(Hkv, 1, dh)
            v = v + t(p + "bv").view(Hkv, 1, dh)
        q, k, v = rnd(q), rnd(k), rnd(v)
        k = k.repeat_interleave(H // Hkv, 0)
        v = v.repeat_interleave(H // Hkv, 0)
        o = F.scaled_dot_product_attention(q[None], k[None], v[None], is_causal=False)[0]
        o = rnd(o.transpose(0, 1).reshape(S, H * dh))
        r = r + o @ t(p + "wo").T
        u2 = rnd(F.rms_norm(r, (d,), t(p + "g2"), eps=geom.rms_eps))
        a = rnd(F.silu(u2 @ t(p + "wg").T) * (u2 @ t(p + "wu").T))
        r = r + a @ t(p + "wd").T
    return rnd(F.rms_norm(r, (d,), t("gf"), eps=geom.rms_eps)).numpy()


# Dream-style geometry at test size: head_dim 128, GQA 4/2, q/k/v biases, RoPE base 1e6, eps 1e-6
GQA_BIAS = dataclasses.replace(
    synth.WORKLOADS["c1s"], key="gqa_bias_dh128", batch=1,
    geom=dataclasses.replace(synth.WORKLOADS["c1s"].geom, name="gqa_bias_dh128", n_heads=4, n_kv_heads=2,
                             head_dim=128, d_model=384, d_ffn=768, qkv_bias=True, weight_dtype="bf16",
                             rope_base=1e6, rms_eps=1e-6))


def _case(tiny_weights, key):
    if key != "gqa_bias_dh128":
        w, stored, _ = tiny_weights(key)
        return w, stored
    return GQA_BIAS, synth.make_weights(GQA_BIAS.geom)


@pytest.mark.parametrize("key", ["c1", "c1s", "gqa_bias_dh128"])
def test_forward_matches_torch_functional_pure(tiny_weights, key):
    """Without the bf16 storage roundings both float64 forwards agree to rounding noise (with q/k/v
    biases and GQA on the Dream-style geometry)."""
    w, stored = _case(tiny_weights, key)
    W = WeightView(stored, bf16_boundary=False)
    tok, p = synth.initial_state(w)
    pos = np.arange(w.seq)
    ours = oracle.forward(w.geom, W, tok[0], pos, bf16_boundary=False)
    ref = _torch_forward(w.geom, W, tok[0], pos, bf16_boundary=False)
    np.testing.assert_allclose(ours, ref, rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("key", ["c1", "c1s", "gqa_bias_dh128"])
def test_forward_matches_torch_functional_bf16(tiny_weights, key):
    """With the storage roundings, an occasional one-ulp flip propagates; rows still agree to a few
    bf16 ulps of their scale."""
    w, stored = _case(tiny_weights, key)
    W = WeightView(stored)
    tok, p = synth.initial_state(w)
    pos = np.arange(w.seq)
    ours = oracle.forward(w.geom, W, tok[0], pos)
    ref = _torch_forward(w.geom, W, tok[0], pos)
    scale = np.abs(ref).max(axis=1, keepdims=True)
    assert (np.abs(ours - ref) <= 2 ** -6 * scale).all()


def test_gqa_with_repeated_kv_equals_mha():
    """A GQA model (H=4, Hkv=2) equals the MHA model whose k/v heads repeat each group's weights."""
    import dataclasses
    g = dataclasses.replace(synth.TINY, n_kv_heads=2, n_layers=1, vocab=512, mask_id=511)
    rng = np.random.default_rng(5)
    d, dh, F_ = g.d_model, g.head_dim, g.d_ffn
    Wd = {"embed": rng.standard_normal((512, d)) * 0.5, "gf": np.ones(d), "l0.g1": np.ones(d),
          "l0.g2": np.ones(d), "l0.wq": rng.standard_normal((4 * dh, d)) * 0.1,
          "l0.wk": rng.standard_normal((2 * dh, d)) * 0.1, "l0.wv": rng.standard_normal((2 * dh, d)) * 0.1,
          "l0.wo": rng.standard_normal((d, 4 * dh)) * 0.05, "l0.wg": rng.standard_normal((F_, d)) * 0.05,
          "l0.wu": rng.standard_normal((F_, d)) * 0.05, "l0.wd": rng.standard_normal((d, F_)) * 0.05}
    gm = dataclasses.replace(g, n_kv_heads=4)
    Wm = dict(Wd)
    rep = lambda w: np.repeat(w.reshape(2, dh, d), 2, axis=0).reshape(4 * dh, d)
    Wm["l0.wk"], Wm["l0.wv"] = rep(Wd["l0.wk"]), rep(Wd["l0.wv"])
    tok = rng.integers(0, 512, 40)
    a = oracle.forward(g, Wd, tok, np.arange(40), bf16_boundary=False)
    b = oracle.forward(gm, Wm, tok, np.arange(40), bf16_boundary=False)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)


def test_permutation_equivariance_without_rope(tiny_weights):
    """Without RoPE the forward is permutation-equivariant: permuting the draft tokens leaves every
    masked row's statistics unchanged (Section 3.3 drafts act only as bidirectional context)."""
    w, stored, W = tiny_weights("c1s")
    tok, p = synth.initial_state(w)
    tok = tok[:1]
    st0 = oracle.step(w.geom, W, tok, p[:1], w.gen_end, rope=False)
    perm = np.random.default_rng(7).permutation(np.arange(48, 64))
    tok2 = tok.copy()
    tok2[0, 48:64] = tok[0, perm]
    st1 = oracle.step(w.geom, W, tok2, p[:1], w.gen_end, rope=False)
    m = st0["conf"][0] >= 0
    np.testing.assert_array_equal(st0["top1"][0, m], st1["top1"][0, m])
    np.testing.assert_allclose(st0["conf"][0, m], st1["conf"][0, m], rtol=1e-9)
    # and with RoPE the draft order does matter
    st2 = oracle.step(w.geom, W, tok2, p[:1], w.gen_end)
    st3 = oracle.step(w.geom, W, tok, p[:1], w.gen_end)
    assert np.abs(st2["conf"][0, m] - st3["conf"][0, m]).max() > 1e-6


def test_kv_prefix_forward_equals_full_forward(tiny_weights):
    """Queries attending to a cache of the prefix's keys/values (as computed in the full bidirectional
    forward) reproduce the full forward's rows exactly."""
    w, stored, W = tiny_weights("c1s")
    tok, _ = synth.initial_state(w)
    P = 48
    full, kvs = oracle.forward(w.geom, W, tok[0], np.arange(w.seq), return_kv=True)
    cache = [(k[:, :P], v[:, :, :P]) for k, v in kvs]
    part = oracle.forward(w.geom, W, tok[0, P:], P + np.arange(w.seq - P), kv=lambda l: cache[l])
    np.testing.assert_array_equal(part, full[P:])


def test_coordinate_permutation_is_a_symmetry(tiny_weights):
    """The whole-step tolerance samples float32 summation orders by permuting the model's d_model and
    d_ffn coordinates. That must be an exact symmetry: the permuted model's hidden states are the
    plain model's with their coordinates permuted, and its step statistics are the same."""
    from helpers import permuted_weights
    w, stored, W = tiny_weights("c1")
    tok, p = synth.initial_state(w)
    pos = np.arange(w.seq)
    Wp = permuted_weights(WeightView(stored, bf16_boundary=False), w.geom, 5)
    pd = np.random.default_rng(5).permutation(w.geom.d_model)
    a = oracle.forward(w.geom, WeightView(stored, bf16_boundary=False), tok[0], pos, bf16_boundary=False)
    b = oracle.forward(w.geom, Wp, tok[0], pos, bf16_boundary=False)
    np.testing.assert_allclose(b, a[:, pd], rtol=1e-10, atol=1e-12)
    s0 = oracle.step(w.geom, W, tok, p, w.gen_end)
    s1 = oracle.step(w.geom, permuted_weights(W, w.geom, 5), tok, p, w.gen_end)
    np.testing.assert_array_equal(s0["top1"], s1["top1"])
    np.testing.assert_allclose(s0["conf"], s1["conf"], rtol=1e-9, atol=1e-12)


def test_bias_enters_before_the_rotation():
    """The q/k biases belong to the projection that RoPE rotates. The torch opinion with the biases added
    after the rotation is a different function, far outside the 1e-10 agreement of the pure-mode pin,
    so that pin rejects the wrong order."""
    w = GQA_BIAS
    stored = synth.make_weights(w.geom)
    W = WeightView(stored, bf16_boundary=False)
    tok, _ = synth.initial_state(w)
    pos = np.arange(w.seq)
    ours = oracle.forward(w.geom, W, tok[0], pos, bf16_boundary=False)
    wrong = _torch_forward(w.geom, W, tok[0], pos, bf16_boundary=False, bias_after_rope=True)
    assert np.abs(ours - wrong).max() > 1e-3


def test_lm_logits_chunking_equals_one_product():
    """lm_logits walks the vocabulary in chunks; with V larger than the chunk (and a ragged last chunk)
    it equals one unchunked product h_f W^T."""
    rng = np.random.default_rng(11)
    V, d = 20011, 64
    Wl = rng.standard_normal((V, d))
    hf = rng.standard_normal((9, d))
    ref = hf @ Wl.T
    for chunk in (8192, 7, V, 3 * V):
        np.testing.assert_allclose(oracle.lm_logits({"lm_head": Wl}, hf, chunk=chunk), ref, rtol=1e-12, atol=1e-12)
    # through the lazy bf16 weight view (uint16 bit patterns widened exactly)
    bits = synth.normal_bf16(5, 0, 0.5, (V, d))
    view = WeightView({"lm_head": bits})
    np.testing.assert_allclose(oracle.lm_logits(view, hf), hf @ synth.bf16_bits_to_f32(bits).astype(np.float64).T,
                               rtol=1e-12, atol=1e-12)


def test_float32_evaluation_runs_in_float32():
    """The float32 evaluation that sizes tolerances must keep float32 arithmetic end to end, RMSNorm
    included: its RMSNorm differs from the float64 one by float32 rounding, not by zero."""
    rng = np.random.default_rng(12)
    r = (rng.standard_normal((64, 512)) * 3).astype(np.float32)
    g = np.ones(512, np.float32)
    a = rmsnorm(r, g, 1e-5)
    assert a.dtype == np.float32
    b = rmsnorm(r.astype(np.float64), g, 1e-5)
    d = np.abs(a - b).max()
    assert 0 < d < 1e-5 * np.abs(b).max()
