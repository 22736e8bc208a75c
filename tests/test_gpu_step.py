"""GPU parity of dcl_denoise_step / dcl_score_hidden (+ dcl_select_contiguous) against the float64
oracle at sizes the oracle finishes in seconds; the shapes span several GEMM, attention and
vocabulary tiles and ragged tails. The bars are described in helpers.py."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from oracle.numerics import WeightView

from helpers import (CONF_TOL, LOGIT_TOL, TIE_GAP, compare_stats, derived_tolerance, runner_for, stats_to_np,
                     to_dev)

pytestmark = pytest.mark.gpu

_W = synth.WORKLOADS


def _variant(name, base, geom_kw, **wl_kw):
    g = dataclasses.replace(base.geom, name=name, **geom_kw)
    return dataclasses.replace(base, key=name, geom=g, **wl_kw)


CASES = {
    "c1": _W["c1"],
    "c1s": _W["c1s"],
    # bf16 weights, head_dim 128, GQA 4/2 with q/k/v bias (Dream-style), B=3
    "gqa_bias_dh128": _variant("gqa_bias_dh128", _W["c1s"],
                               dict(n_heads=4, n_kv_heads=2, head_dim=128, d_model=384, d_ffn=768, qkv_bias=True,
                                    weight_dtype="bf16", rope_base=1e6, rms_eps=1e-6), batch=3),
    # ragged everything: S=77, d=208 (K tail 16), F=400, vocab 1000 (last vocab tile 104 ids), H*dh != d
    "ragged": _variant("ragged", _W["c1s"],
                       dict(n_heads=2, n_kv_heads=1, head_dim=64, d_model=208, d_ffn=400, vocab=1000, mask_id=999),
                       batch=2, prompt_len=29, gen_len=48, window=16, p=29, draft=(45, 61)),
    # 48 tokens: a single 64-key tile, so the second key group of the attention has no keys (on the
    # well-conditioned tiny model: the spread one turns rare bf16 rounding flips into lse changes
    # several times its float32 drift at this length, with either attention path)
    "short": _variant("short", _W["c1"], {}, batch=2, prompt_len=16, gen_len=32, window=16, p=16, draft=(24, 40)),
    # 16 x 16 heads x 256 tokens = 4096 query waves: the attention path with one key group of
    # 8 query waves (head_dim 64, GQA 16/4, H*dh != d)
    "many_heads": _variant("many_heads", _W["c1s"],
                           dict(n_layers=1, n_heads=16, n_kv_heads=4, head_dim=64, d_model=512, d_ffn=512,
                                vocab=1000, mask_id=999),
                           batch=16, prompt_len=64, gen_len=192, window=32, p=64, draft=(128, 192)),
    # vocabulary 50001 at 192 rows: the LM head runs 256-id workgroup tiles whose two waves each own
    # a 128-id vocabulary tile; 391 tiles, the last one 81 ids wide, the last workgroup's second
    # wave past the end
    "vocab_50001": _variant("vocab_50001", _W["c1"], dict(vocab=50001, mask_id=50000), batch=2),
    # larger tile counts: S=320 (5 query tiles), vocab 8192, 3 layers
    "wide": _variant("wide", _W["c1s"], dict(n_layers=3, d_model=512, n_heads=8, n_kv_heads=8, d_ffn=1376,
                                             vocab=8192, mask_id=8191, weight_dtype="bf16"),
                     batch=1, prompt_len=96, gen_len=224, window=32, p=96, draft=(128, 192)),
    # full LLaDA-8B width and vocabulary, 2 of its 32 layers: the tile plans and split-K of the
    # 384-token step (B1, 128 prompt + 256 generation), the 126464-id LM head
    "llada_2l": _variant("llada_2l", _W["c2"], dict(n_layers=2)),
    # full Dream-7B width and vocabulary (GQA 28/4, biases), 2 of 28 layers, B2 x 384 tokens
    "dream_2l": _variant("dream_2l", _W["c4"], dict(n_layers=2), batch=2, prompt_len=128, gen_len=256),
}

_cache = {}


def _setup(key):
    if key not in _cache:
        w = CASES[key]
        stored = synth.make_weights(w.geom)
        _cache[key] = (w, stored, WeightView(stored), runner_for(w, stored))
    return _cache[key]


@pytest.mark.parametrize("key", list(CASES))
def test_step_parity(key):
    w, stored, W, run = _setup(key)
    print(f"case {key}: B={w.batch} S={w.seq} geom={w.geom.name}", flush=True)
    tok, p = synth.initial_state(w)
    ref = oracle.step(w.geom, W, tok, p, w.gen_end)
    ct, lt = derived_tolerance(w.geom, W, tok, p, w.gen_end, ref)
    st = run.step(to_dev(tok), to_dev(p), w.gen_end)
    compare_stats(stats_to_np(st), ref, w.tau_commit, w.tau_draft, what=key, conf_tol=ct, logit_tol=lt)


@pytest.mark.parametrize("key", ["c1", "c1s", "ragged", "gqa_bias_dh128", "wide", "vocab_50001", "llada_2l"])
def test_lm_head_on_gpu_hidden_exact_bar(key):
    """Exact-input stage: the GPU's float32 logits equal h_f W_lm^T (float64) of the GPU's own bf16 final
    hidden states within 2e-2, and those hidden states stay close to the oracle's."""
    import torch
    w, stored, W, run = _setup(key)
    tok, p = synth.initial_state(w)
    B, S = tok.shape
    rows = np.array(sorted(set([0, S - 1, w.p, w.p + 1, S * (B - 1) + w.p, B * S - 1])), np.int64)
    got, hid = run.logits(to_dev(tok), torch.from_numpy(rows.astype(np.int32)).cuda(), with_hidden=True)
    got = got.cpu().numpy()
    h = synth.bf16_bits_to_f32(hid.cpu().numpy().view(np.uint16)).astype(np.float64)
    exact = oracle.lm_logits(W, h)
    err = np.abs(got - exact).max()
    ref = oracle.step(w.geom, W, tok, p, w.gen_end, return_logits_rows=rows, return_hidden=True)
    href = ref["hidden"].reshape(B * S, -1)[rows]
    rel = np.abs(h - href).max(axis=1) / np.abs(href).max(axis=1)
    print(key, "logit max-abs vs exact LM head", err, "| hidden: elements equal %.3f, max rel-to-row-scale %.3g"
          % ((h == href).mean(), rel.max()), "| logit max-abs vs oracle", np.abs(got - ref["logits"]).max(), flush=True)
    assert err <= LOGIT_TOL
    assert rel.max() < 0.1


@pytest.mark.parametrize("key", ["c1", "ragged", "wide", "llada_2l", "dream_2l"])
def test_score_hidden_exact_bar(key):
    """dcl_score_hidden (fused LM head + vocabulary reduction) on synthetic bf16 hidden rows vs the oracle's
    materialised softmax: conf within 1e-3, lse within 2e-2, ids exact except near-ties."""
    import torch
    w, stored, W, run = _setup(key)
    n = 203
    h = synth.normal_bf16(77, 0, 1.0, (n, w.geom.d_model))
    st = stats_to_np(run.score_hidden(torch.from_numpy(h.view(np.int16)).cuda()))
    lg = oracle.lm_logits(W, synth.bf16_bits_to_f32(h).astype(np.float64))
    t1, t2, c, p2, lse = oracle.row_stats(lg)
    H = oracle.row_entropy(lg)
    ref = {"top1": t1[None], "top2": t2[None], "conf": c[None], "p2": p2[None], "lse": lse[None], "entropy": H[None]}
    gpu = {k: v[None] for k, v in st.items()}
    # entropy bar per row: dH/dl_v = -P_v (l_v - E_P l), so |dH| <= max|dl| * E_P|l - E_P l| <= max|dl| * sd_P(l)
    P = np.exp(lg - lse[:, None])
    sd = np.sqrt(np.maximum((P * lg ** 2).sum(1) - (P * lg).sum(1) ** 2, 0.0))
    rep = compare_stats(gpu, ref, what=f"score_hidden[{key}]", entropy_tol=(LOGIT_TOL * np.maximum(sd, 1.0))[None])
    assert rep["meets_exact_input_bar"]
    np.testing.assert_allclose(st["p2"], p2, atol=CONF_TOL)
    gap = np.log(c) - np.log(p2)
    ok = gap >= TIE_GAP
    np.testing.assert_array_equal(st["top2"][ok & (st["top1"] == t1)], t2[ok & (st["top1"] == t1)])


def test_score_all_uncommitted_mode():
    import paper_2607_20467_amd as dcl
    w, stored, W, run = _setup("c1s")
    tok, p = synth.initial_state(w)
    ref = oracle.step(w.geom, W, tok, p, w.gen_end, score_all=True)
    ct, lt = derived_tolerance(w.geom, W, tok, p, w.gen_end, ref, score_all=True)
    st = run.step(to_dev(tok), to_dev(p), w.gen_end, flags=dcl.DCL_SCORE_ALL_UNCOMMITTED)
    compare_stats(stats_to_np(st), ref, w.tau_commit, w.tau_draft, what="score_all", conf_tol=ct, logit_tol=lt)


def test_rope_disabled_matches_oracle():
    w, stored, W, _ = _setup("c1s")
    run = runner_for(w, stored, rope=False)
    tok, p = synth.initial_state(w)
    ref = oracle.step(w.geom, W, tok, p, w.gen_end, rope=False)
    ct, lt = derived_tolerance(w.geom, W, tok, p, w.gen_end, ref, rope=False)
    compare_stats(stats_to_np(run.step(to_dev(tok), to_dev(p), w.gen_end)), ref, w.tau_commit, what="no-rope",
                  conf_tol=ct, logit_tol=lt)


def test_kv_prefix_step():
    """Queries attend to [cached prefix || fresh tokens]: tiny analogue of the 1216-token prefix case."""
    import torch
    base = CASES["c1s"]
    w = dataclasses.replace(base, key="kv", batch=2, prompt_len=0, gen_len=32, window=16, p=0, draft=(16, 32),
                            kv_prefix=64, kv_seed=3)
    stored = _setup("c1s")[1]
    W = WeightView(stored)
    run = runner_for(w, stored)
    caches = [synth.kv_cache_layer(w, l) for l in range(w.geom.n_layers)]

    def kv(b, l):
        k, v = caches[l]
        return synth.bf16_bits_to_f32(k[b]), synth.bf16_bits_to_f32(v[b])
    kv.prefix = w.kv_prefix
    tok, p = synth.initial_state(w)
    ref = oracle.step(w.geom, W, tok, p, w.gen_end, kv=kv)
    ct, lt = derived_tolerance(w.geom, W, tok, p, w.gen_end, ref, kv=kv)
    ks = [torch.from_numpy(c[0].view(np.int16)).cuda() for c in caches]
    vs = [torch.from_numpy(c[1].view(np.int16)).cuda() for c in caches]
    st = run.step(to_dev(tok), to_dev(p), w.gen_end, kv=(ks, vs, w.kv_prefix))
    compare_stats(stats_to_np(st), ref, w.tau_commit, w.tau_draft, what="kv-prefix", conf_tol=ct, logit_tol=lt)


def test_step_is_deterministic():
    w, stored, W, run = _setup("wide")
    tok, p = synth.initial_state(w)
    a = stats_to_np(run.step(to_dev(tok), to_dev(p), w.gen_end))
    for _ in range(3):
        b = stats_to_np(run.step(to_dev(tok), to_dev(p), w.gen_end))
        for k in a:
            np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def test_full_loop_matches_oracle_every_iteration():
    """Algorithm 1 end to end with device-resident tokens and p: at every iteration the GPU statistics
    are checked against the oracle on the same state, and the GPU selection must equal the oracle's
    selection rule applied to the GPU statistics (bit-exact). Whole trajectories are not compared:
    one rounding-level confidence difference at a threshold legitimately changes the path."""
    import paper_2607_20467_amd as dcl
    w, stored, W, run = _setup("c1s")
    prompt = synth.prompts(w)
    M, L, tc, td = 48, 16, 0.7, 0.9
    N = prompt.shape[1]
    x = np.concatenate([prompt, np.full((prompt.shape[0], M), w.geom.mask_id)], 1).astype(np.int32)
    tok = to_dev(x)
    p = to_dev(np.full(prompt.shape[0], N, np.int32))
    B, S = x.shape
    st = run.new_stats(B, S)
    n = 0
    p_host = p.cpu().numpy()
    # tolerance sized once on the full initial state (96 scored rows): the drift of a late state with
    # only a few scored rows is too small a sample to bound the GPU's
    ref0 = oracle.step(w.geom, W, x, p_host, S)
    ct, lt = derived_tolerance(w.geom, W, x, p_host, S, ref0)
    while (p_host < S).any():
        assert n < M, "loop exceeded M iterations"
        x_before, p_before = tok.cpu().numpy(), p_host
        run.step(tok, p, S, stats=st)
        g = stats_to_np(st)
        ref = oracle.step(w.geom, W, x_before, p_before, S)
        compare_stats(g, ref, tc, td, what=f"iteration {n}", conf_tol=ct, logit_tol=lt)
        dcl.dcl_select_contiguous(tok, B, S, p, S, L, tc, td, w.geom.mask_id, st)
        x_ref, p_ref, _, _ = oracle.select_contiguous(x_before, p_before, S, L, tc, td, w.geom.mask_id, g["top1"],
                                                      g["conf"].astype(np.float64))
        p_host = p.cpu().numpy()
        np.testing.assert_array_equal(tok.cpu().numpy(), x_ref)
        np.testing.assert_array_equal(p_host, p_ref)
        assert (p_host > p_before)[p_before < S].all()
        n += 1
    print("loop finished in", n, "iterations", flush=True)


def test_mask_suppression_step():
    """DCL_SCORE_SUPPRESS_MASK: the LM-head row of [MASK] is steered (through the oracle's own hidden
    states) so that [MASK] would be the top-1 of every scored row; with the flag the statistics match
    the oracle's softmax over the vocabulary without that id, and [MASK] is never top-1 or top-2."""
    import paper_2607_20467_amd as dcl
    w = CASES["c1"]
    stored = dict(synth.make_weights(w.geom))
    tok, p = synth.initial_state(w)
    ref0 = oracle.step(w.geom, WeightView(stored), tok, p, w.gen_end, return_hidden=True)
    sc = ref0["conf"] >= 0
    hs = ref0["hidden"][sc]
    d = (hs / np.linalg.norm(hs, axis=1, keepdims=True)).sum(0)
    lm = stored["lm_head"].copy()
    lm[w.geom.mask_id] = (d / np.linalg.norm(d) * np.linalg.norm(lm, axis=1).mean() * 3).astype(lm.dtype)
    stored["lm_head"] = lm
    W = WeightView(stored)
    run = runner_for(w, stored)
    plain = oracle.step(w.geom, W, tok, p, w.gen_end)
    assert (plain["top1"][sc] == w.geom.mask_id).mean() > 0.9     # the steering worked
    ref = oracle.step(w.geom, W, tok, p, w.gen_end, suppress_mask=True)
    ct, lt = derived_tolerance(w.geom, W, tok, p, w.gen_end, ref, suppress_mask=True)
    g = stats_to_np(run.step(to_dev(tok), to_dev(p), w.gen_end, flags=dcl.DCL_SCORE_SUPPRESS_MASK))
    assert not (g["top1"][sc] == w.geom.mask_id).any() and not (g["top2"][sc] == w.geom.mask_id).any()
    compare_stats(g, ref, what="suppress", conf_tol=ct, logit_tol=lt)
    # and without the flag the GPU follows the unsuppressed oracle
    ct0, lt0 = derived_tolerance(w.geom, W, tok, p, w.gen_end, plain)
    compare_stats(stats_to_np(run.step(to_dev(tok), to_dev(p), w.gen_end)), plain, what="plain", conf_tol=ct0,
                  logit_tol=lt0)


def test_entropy_of_steered_and_flat_rows():
    """Entropy through the fused reduction at its extremes: a hidden row aligned with one LM-head row
    (near one-hot, H -> 0) and the zero hidden row (uniform softmax, H = log V exactly)."""
    import torch
    w, stored, W, run = _setup("c1")
    V, d = w.geom.vocab, w.geom.d_model
    lm = np.asarray(stored["lm_head"], np.float32)
    h = np.zeros((2, d), np.float32)
    h[0] = lm[17] / np.linalg.norm(lm[17]) * 8.0
    hb = torch.from_numpy(h).to(torch.bfloat16)
    st = stats_to_np(run.score_hidden(hb.view(torch.int16).cuda()))
    lg = oracle.lm_logits(W, hb.float().numpy().astype(np.float64))
    H = oracle.row_entropy(lg)
    print("entropy: steered row", st["entropy"][0], "oracle", H[0], "| zero row", st["entropy"][1], "log V", np.log(V))
    assert H[1] == pytest.approx(np.log(V), rel=1e-12)
    assert abs(st["entropy"][1] - np.log(V)) < 1e-4
    assert abs(st["entropy"][0] - H[0]) < 2 * LOGIT_TOL


@pytest.mark.parametrize("key,B,P,S,cap", [("gqa_bias_dh128", 3, 40, 21, 48), ("dream_2l", 2, 72, 27, 80)])
def test_kv_prefix_step_ragged_gqa_with_spare_capacity(key, B, P, S, cap):
    """A prefix that is not a multiple of 64 keys (a 64-key tile then holds cache and fresh keys),
    fresh tokens not a multiple of 8, GQA with head_dim 128 and q/k/v bias (a small model, and two
    layers of the Dream-7B geometry: 28/4 heads, d 3584, vocabulary 152064), and a cache whose
    capacity exceeds the prefix: the unused positions hold large finite values that must never be
    read."""
    import torch
    base = CASES[key]
    w = dataclasses.replace(base, key="kv_ragged_" + key, batch=B, prompt_len=0, gen_len=S, window=8, p=0,
                            draft=(8, 16), kv_prefix=P, kv_seed=5)
    stored = _setup(key)[1]
    W = WeightView(stored)
    run = runner_for(w, stored)
    g = w.geom
    caches = [synth.kv_cache_layer(w, l) for l in range(g.n_layers)]

    def kv(b, l):
        k, v = caches[l]
        return synth.bf16_bits_to_f32(k[b]), synth.bf16_bits_to_f32(v[b])
    kv.prefix = w.kv_prefix
    tok, p = synth.initial_state(w)
    ref = oracle.step(g, W, tok, p, w.gen_end, kv=kv)
    ct, lt = derived_tolerance(g, W, tok, p, w.gen_end, ref, kv=kv)
    big = np.uint16(0x4700)                          # bf16 32768
    ks, vs = [], []
    for k, v in caches:
        kk = np.full((w.batch, g.n_kv_heads, cap, g.head_dim), big, np.uint16)
        vv = np.full((w.batch, g.n_kv_heads, g.head_dim, cap), big, np.uint16)
        kk[:, :, :P] = k
        vv[:, :, :, :P] = v
        ks.append(torch.from_numpy(kk.view(np.int16)).cuda())
        vs.append(torch.from_numpy(vv.view(np.int16)).cuda())
    st = run.step(to_dev(tok), to_dev(p), w.gen_end, kv=(ks, vs, P, cap))
    compare_stats(stats_to_np(st), ref, w.tau_commit, w.tau_draft, what="kv-prefix-ragged", conf_tol=ct, logit_tol=lt)
