"""GPU parity of dcl_denoise_step (+ dcl_select_contiguous) against the float64 oracle at sizes the
oracle finishes in seconds; they span several GEMM / attention / vocabulary tiles and ragged tails."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from oracle.numerics import WeightView

from helpers import LOGIT_TOL, compare_stats, runner_for, stats_to_np, to_dev

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
    # larger tile counts: S=320 (5 query tiles), vocab 8192, 3 layers
    "wide": _variant("wide", _W["c1s"], dict(n_layers=3, d_model=512, n_heads=8, n_kv_heads=8, d_ffn=1376,
                                             vocab=8192, mask_id=8191, weight_dtype="bf16"),
                     batch=1, prompt_len=96, gen_len=224, window=32, p=96, draft=(128, 192)),
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
    st = run.step(to_dev(tok), to_dev(p), w.gen_end)
    compare_stats(stats_to_np(st), ref, w.tau_commit, w.tau_draft, what=key)


@pytest.mark.parametrize("key", ["c1", "c1s", "ragged", "gqa_bias_dh128"])
def test_logits_parity(key):
    """float32 logits of the bf16 model vs float64 oracle logits (max-abs 2e-2), incl. unscored rows."""
    import torch
    w, stored, W, run = _setup(key)
    tok, p = synth.initial_state(w)
    B, S = tok.shape
    rows = np.array(sorted(set([0, S - 1, w.p, w.p + 1, S * (B - 1) + w.p, B * S - 1])), np.int64)
    ref = oracle.step(w.geom, W, tok, p, w.gen_end, return_logits_rows=rows)["logits"]
    got = run.logits(to_dev(tok), torch.from_numpy(rows.astype(np.int32)).cuda()).cpu().numpy()
    err = np.abs(got - ref).max()
    print(key, "logit max-abs", err, "max |logit|", np.abs(ref).max(), flush=True)
    assert err <= LOGIT_TOL


def test_score_all_uncommitted_mode():
    w, stored, W, run = _setup("c1s")
    import paper_2607_20467_amd as dcl
    tok, p = synth.initial_state(w)
    ref = oracle.step(w.geom, W, tok, p, w.gen_end, score_all=True)
    st = run.step(to_dev(tok), to_dev(p), w.gen_end, flags=dcl.DCL_SCORE_ALL_UNCOMMITTED)
    compare_stats(stats_to_np(st), ref, w.tau_commit, w.tau_draft, what="score_all")


def test_rope_disabled_matches_oracle():
    w, stored, W, _ = _setup("c1s")
    run = runner_for(w, stored, rope=False)
    tok, p = synth.initial_state(w)
    ref = oracle.step(w.geom, W, tok, p, w.gen_end, rope=False)
    compare_stats(stats_to_np(run.step(to_dev(tok), to_dev(p), w.gen_end)), ref, w.tau_commit, what="no-rope")


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
    ks = [torch.from_numpy(c[0].view(np.int16)).cuda() for c in caches]
    vs = [torch.from_numpy(c[1].view(np.int16)).cuda() for c in caches]
    st = run.step(to_dev(tok), to_dev(p), w.gen_end, kv=(ks, vs, w.kv_prefix))
    compare_stats(stats_to_np(st), ref, w.tau_commit, w.tau_draft, what="kv-prefix")


def test_step_is_deterministic():
    import torch
    w, stored, W, run = _setup("wide")
    tok, p = synth.initial_state(w)
    a = stats_to_np(run.step(to_dev(tok), to_dev(p), w.gen_end))
    for _ in range(3):
        b = stats_to_np(run.step(to_dev(tok), to_dev(p), w.gen_end))
        for k in a:
            np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def test_full_loop_matches_oracle():
    """Algorithm 1 end to end: device-resident tokens and p, one step + one select per iteration."""
    import torch
    import paper_2607_20467_amd as dcl
    w, stored, W, run = _setup("c1s")
    prompt = synth.prompts(w)
    M, L, tc, td = 48, 16, 0.7, 0.9
    N = prompt.shape[1]
    ref, steps = oracle.generate(w.geom, W, prompt, M, L, tc, td)
    x = np.concatenate([prompt, np.full((prompt.shape[0], M), w.geom.mask_id)], 1).astype(np.int32)
    tok = to_dev(x)
    p = to_dev(np.full(prompt.shape[0], N, np.int32))
    B, S = x.shape
    st = run.new_stats(B, S)
    n = 0
    while (p.cpu().numpy() < S).any():
        assert n < M
        run.step(tok, p, S, stats=st)
        dcl.dcl_select_contiguous(tok, B, S, p, S, L, tc, td, w.geom.mask_id, st)
        n += 1
    print("loop steps gpu", n, "oracle", steps, flush=True)
    np.testing.assert_array_equal(tok.cpu().numpy(), ref)
    assert n == steps
