"""Stage-wise parity of the transformer forward at the full shapes of the 7-8B workloads (c2-c5), every
layer, plus the fused LM head on its production tile plans.

Forward (rows a3-a8, a14): the GPU's residual stream is teacher-forced through the layers with
dcl_debug_layer (the step's own kernels, plans and split-K folding). At every layer each stage is fed
the GPU's own input of that stage, on both sides:

  u     = bf16(RMSNorm(r_in) g1)                 oracle.forward.norm_stage
  q,k,v = bf16(RoPE(u W^T + b))                  oracle.forward.qkv_stage
  o     = bf16(softmax(q k^T / sqrt(dh)) v)      oracle.forward.attention_stage (GQA, cached prefix)
  r_mid = r_in + o W_o^T                         oracle.forward.residual_stage (split-K slices folded)
  u2    = bf16(RMSNorm(r_mid) g2)
  a     = bf16(silu(u2 W_g^T) (u2 W_u^T))         oracle.forward.swiglu_stage
  r_out = r_mid + a W_d^T

and compared element by element on sampled token rows against a float32 error bound derived for that
stage (stage_checks.py). The final norm h_f = bf16(RMSNorm(r_L) g_f) of the scored rows is checked the
same way on the chained r_L, which also shows the chain reproduces the step's own hidden states.

LM head (rows a9, a10, f4): the step's statistics (its fused LM-head epilogue on the production plan
of that token count) against the oracle's statistics of the step's own final hidden states, at the
exact-input bar: confidences within 1e-3, log-sum-exp within 2e-2, top-1 ids identical except near-ties,
entropy within the derived per-row bar. dcl_score_hidden runs the same check at the token counts whose
tuned plans have every wave own a 128-id vocabulary tile.
"""
import dataclasses
import time

import numpy as np
import pytest

import oracle
import synth
from oracle.forward import attention_stage, norm_stage, qkv_stage, residual_stage, swiglu_stage
from oracle.numerics import WeightView, rope_tables

import stage_checks as sc
from helpers import CONF_TOL, LOGIT_TOL, TIE_GAP, compare_stats, full_runner, runner_for, stats_to_np, to_dev

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

ROWS = 24            # sampled token rows per workload and layer (plus the first and last of each sequence)
HEAD_ROWS = 512      # scored rows whose LM-head statistics are recomputed by the oracle (all if fewer)
_ident = lambda a: a


def _layer_weights(view, geom, l):
    names = ["wq", "wk", "wv", "wo", "wg", "wu", "wd", "g1", "g2"] + (["bq", "bk", "bv"] if geom.qkv_bias else [])
    return {f"l{l}.{n}": view(f"l{l}.{n}") for n in names}


class _Case:
    """GPU-side state of one workload: decode state, cache, the residual stream and the tap buffers."""

    def __init__(self, w, run, stored):
        import torch
        w = synth.WORKLOADS[w] if isinstance(w, str) else w
        self.key, self.w, self.run = w.key, w, run
        w, g = self.w, self.w.geom
        self.tok, self.p = synth.initial_state(w)
        self.B, self.S = self.tok.shape
        self.P = w.kv_prefix
        self.T, self.Sp = self.B * self.S, (self.P % 8 + self.S + 7) // 8 * 8
        self.kv_host = None
        self.kv = None
        if self.P:
            self.kv_host = [synth.kv_cache_layer(w, l) for l in range(g.n_layers)]
            cap = (self.P + 7) // 8 * 8       # cache capacity: positions [0, P) in use

            def pad(x, axis):
                shape = list(x.shape)
                shape[axis] = cap
                out = np.zeros(shape, x.dtype)
                out[(slice(None),) * axis + (slice(0, self.P),)] = x
                return torch.from_numpy(out.view(np.int16)).cuda()
            self.kv = ([pad(c[0], 2) for c in self.kv_host], [pad(c[1], 3) for c in self.kv_host], self.P, cap)
        self.t_dev, self.p_dev = to_dev(self.tok), to_dev(self.p)
        emb = synth.bf16_bits_to_f32(stored["embed"][self.tok])          # r_0 = E[x] widened exactly
        self.r = torch.from_numpy(emb.reshape(self.T, g.d_model)).cuda()
        d, F, hd, kd = g.d_model, g.d_ffn, g.n_heads * g.head_dim, g.n_kv_heads * g.head_dim
        i16, f32 = torch.int16, torch.float32
        self.taps = {"u": torch.empty(self.T * d, dtype=i16, device="cuda"),
                     "q": torch.empty(self.T * hd, dtype=i16, device="cuda"),
                     "k": torch.empty(self.B * (self.P % 8 + self.S) * kd, dtype=i16, device="cuda"),
                     "v": torch.empty(self.B * kd * self.Sp, dtype=i16, device="cuda"),
                     "o": torch.empty(self.T * hd, dtype=i16, device="cuda"),
                     "r_mid": torch.empty(self.T * d, dtype=f32, device="cuda"),
                     "u2": torch.empty(self.T * d, dtype=i16, device="cuda"),
                     "a": torch.empty(self.T * F, dtype=i16, device="cuda"),
                     "r_out": torch.empty(self.T * d, dtype=f32, device="cuda")}
        self.cos, self.sin = rope_tables(self.P + np.arange(self.S), g.head_dim, g.rope_base)
        self.reports = []

    def sample_rows(self, l):
        rng = np.random.default_rng([self.w.geom.seed, 500 + l, self.T])
        pick = {0, self.T - 1}
        for b in range(self.B):
            pick |= {b * self.S, b * self.S + self.S - 1, b * self.S + int(self.p[b])}
        pick |= set(rng.choice(self.T, min(ROWS, self.T), replace=False).tolist())
        return np.array(sorted(pick))


def _layer_step(case, l, Wl):
    """Run layer l of the chain on the GPU and check every stage on sampled rows."""
    import torch
    import paper_2607_20467_amd as dcl
    w, g = case.w, case.w.geom
    H, Hkv, dh, d, F = g.n_heads, g.n_kv_heads, g.head_dim, g.d_model, g.d_ffn
    ws, n = case.run.workspace(case.B, case.S, case.P)
    dcl.dcl_debug_layer(case.run.model, case.B, case.S, case.kv, l, case.r, case.taps, ws, n)
    rows = case.sample_rows(l)
    bs, ss = rows // case.S, rows % case.S
    rows_t = torch.from_numpy(rows).cuda()
    host = lambda name, width: case.taps[name].view(case.T, width)[rows_t].cpu().numpy()
    r_in = case.r[rows_t].cpu().numpy().astype(np.float64)
    u = host("u", d)
    r_mid = host("r_mid", d).astype(np.float64)
    u2 = host("u2", d)
    a = host("a", F)
    r_out = host("r_out", d).astype(np.float64)
    o = host("o", H * dh)
    q_all = case.taps["q"].view(case.B, H, case.S, dh)
    koff = case.P % 8                    # slots of the newest cached keys carried in front of the fresh ones
    k_all = case.taps["k"].view(case.B, Hkv, koff + case.S, dh)[:, :, koff:].cpu().numpy()
    v_all = case.taps["v"].view(case.B, Hkv, dh, case.Sp)[:, :, :, koff:koff + case.S].cpu().numpy()
    q = q_all[torch.from_numpy(bs).cuda(), :, torch.from_numpy(ss).cuda()].cpu().numpy()   # [n, H, dh]
    W = lambda name: Wl[name]
    p_ = f"l{l}."
    rep = {"workload": case.key, "layer": l, "rows": len(rows)}

    # RMSNorm (a3)
    x = norm_stage(r_in, W(p_ + "g1"), g.rms_eps, _ident)
    sc.check_bf16("u", u, x, sc.norm_bound(x, d), rep)
    uf = sc.bf16_bits_to_f64(u)
    # QKV + bias + RoPE (a4)
    cos, sin = case.cos[ss], case.sin[ss]
    qx, kx, vx = qkv_stage(g, W, l, uf, cos, sin, _ident)              # [H, n, dh], [Hkv, n, dh] x2
    ua = np.abs(uf)
    bias = (lambda nm: np.abs(W(p_ + nm))) if g.qkv_bias else (lambda nm: None)
    pre = {}
    for nm, heads, wn, bn in (("q", H, "wq", "bq"), ("k", Hkv, "wk", "bk"), ("v", Hkv, "wv", "bv")):
        E = sc.linear_bound(ua, np.abs(W(p_ + wn)), bias(bn))
        val = uf @ W(p_ + wn).T + (W(p_ + bn) if g.qkv_bias else 0.0)
        pre[nm] = (E.reshape(len(rows), heads, dh).transpose(1, 0, 2), val.reshape(len(rows), heads, dh).transpose(1, 0, 2))
    Eq = sc.rope_pair_bound(*pre["q"], dh // 2)
    Ek = sc.rope_pair_bound(*pre["k"], dh // 2)
    sc.check_bf16("q", q.transpose(1, 0, 2), qx, Eq, rep)
    k_rows = k_all[bs, :, ss]                                            # [n, Hkv, dh]
    v_rows = v_all[bs, :, :, ss]                                         # [n, Hkv, dh]
    sc.check_bf16("k", k_rows.transpose(1, 0, 2), kx, Ek, rep)
    sc.check_bf16("v", v_rows.transpose(1, 0, 2), vx, pre["v"][0], rep)
    # attention (a5; a14 with the cached prefix), per sequence over all of its keys
    scale_log2 = np.log2(np.e) / np.sqrt(dh)
    ex_o = np.empty((len(rows), H * dh))
    E_o = np.empty((len(rows), H * dh))
    qf = sc.bf16_bits_to_f64(q)                                          # [n, H, dh]
    for b in np.unique(bs):
        sel = np.nonzero(bs == b)[0]
        kb = sc.bf16_bits_to_f64(k_all[b])                               # [Hkv, S, dh]
        vb = sc.bf16_bits_to_f64(v_all[b]).transpose(0, 2, 1)
        if case.P:
            kc, vc = case.kv_host[l]                                     # cache buffers; positions [0, P) in use
            kb = np.concatenate([sc.bf16_bits_to_f64(kc[b][:, :case.P]), kb], axis=1)
            vb = np.concatenate([sc.bf16_bits_to_f64(vc[b][:, :, :case.P]).transpose(0, 2, 1), vb], axis=1)
        qb = qf[sel].transpose(1, 0, 2)                                  # [H, m, dh]
        ex_o[sel] = attention_stage(g, qb, kb, vb, _ident)
        for h in range(H):
            kk, vv = kb[h // (H // Hkv)], vb[h // (H // Hkv)]
            s_ = qb[h] @ kk.T / np.sqrt(dh)
            Pm = np.exp(s_ - s_.max(axis=1, keepdims=True))
            Pm /= Pm.sum(axis=1, keepdims=True)
            E_o[sel, h * dh:(h + 1) * dh] = sc.attention_bound(qb[h], kk, vv, Pm, scale_log2)
    sc.check_bf16("o", o, ex_o, E_o, rep)
    # O projection + residual, split-K slices folded (a6)
    of = sc.bf16_bits_to_f64(o)
    Wo = W(p_ + "wo")
    sc.check_f32("r_mid", r_mid, residual_stage(r_in, of, Wo),
                 sc.linear_bound(np.abs(of), np.abs(Wo), np.abs(r_in), extra_terms=4), rep)
    # second RMSNorm, gate/up + SwiGLU (a7)
    x2 = norm_stage(r_mid, W(p_ + "g2"), g.rms_eps, _ident)
    sc.check_bf16("u2", u2, x2, sc.norm_bound(x2, d), rep)
    u2f = sc.bf16_bits_to_f64(u2)
    gate, up = u2f @ W(p_ + "wg").T, u2f @ W(p_ + "wu").T
    Eg = sc.linear_bound(np.abs(u2f), np.abs(W(p_ + "wg")))
    Eu = sc.linear_bound(np.abs(u2f), np.abs(W(p_ + "wu")))
    sc.check_bf16("a", a, swiglu_stage(W, l, u2f, _ident), sc.swiglu_bound(gate, up, Eg, Eu), rep)
    # down projection + residual (a7)
    af = sc.bf16_bits_to_f64(a)
    Wd = W(p_ + "wd")
    sc.check_f32("r_out", r_out, residual_stage(r_mid, af, Wd),
                 sc.linear_bound(np.abs(af), np.abs(Wd), np.abs(r_mid), extra_terms=4), rep)
    case.r.copy_(case.taps["r_out"].view(case.T, d))
    case.reports.append(rep)
    return rep


def _final_and_head(case, view):
    """Final norm of the scored rows on the chained r_L (a8) and the step's LM-head statistics on the
    step's own h_f at the exact-input bar (a9, a10, f4)."""
    import torch
    w, g = case.w, case.w.geom
    st = stats_to_np(case.run.step(case.t_dev, case.p_dev, w.gen_end, kv=case.kv))
    scored = np.nonzero(st["conf"].reshape(-1) >= 0)[0]
    ref_rows = np.nonzero(oracle.scored_mask(case.tok, case.p, w.gen_end, g.mask_id).reshape(-1))[0]
    np.testing.assert_array_equal(scored, ref_rows)
    _, hid = case.run.logits(case.t_dev, torch.from_numpy(scored.astype(np.int32)).cuda(), kv=case.kv,
                             with_hidden=True)
    hid = hid.cpu().numpy()
    rL = case.r[torch.from_numpy(scored).cuda()].cpu().numpy().astype(np.float64)
    x = norm_stage(rL, view("gf"), g.rms_eps, _ident)
    rep = {"workload": case.key, "stage": "final norm + LM head", "scored_rows": len(scored)}
    sc.check_bf16("h_f", hid, x, sc.norm_bound(x, g.d_model), rep)
    # LM head + vocabulary reduction of the step, against the oracle's statistics of the same h_f
    rng = np.random.default_rng([g.seed, 900])
    pick = np.sort(rng.choice(len(scored), min(HEAD_ROWS, len(scored)), replace=False))
    hf = sc.bf16_bits_to_f64(hid[pick])
    lg = oracle.lm_logits(view, hf)
    t1, t2, c, p2, lse = oracle.row_stats(lg)
    ent = oracle.row_entropy(lg)
    flat = lambda k: st[k].reshape(-1)[scored[pick]][None]
    gpu = {k: flat(k) for k in ("top1", "top2", "conf", "p2", "lse", "entropy")}
    ref = {"top1": t1[None], "top2": t2[None], "conf": c[None], "p2": p2[None], "lse": lse[None], "entropy": ent[None]}
    P = np.exp(lg - lse[:, None])
    sd = np.sqrt(np.maximum((P * lg ** 2).sum(1) - (P * lg).sum(1) ** 2, 0.0))
    rep["lm_head"] = compare_stats(gpu, ref, w.tau_commit, w.tau_draft, what=f"{case.key} step LM head on its own h_f",
                                   entropy_tol=(LOGIT_TOL * np.maximum(sd, 1.0))[None])
    assert rep["lm_head"]["meets_exact_input_bar"]
    return rep


def _run_geometry(keys, stored=None, run=None):
    w0 = synth.WORKLOADS[keys[0]] if isinstance(keys[0], str) else keys[0]
    g = w0.geom
    if run is None:
        stored, run = full_runner(w0)
    view = WeightView(stored)
    cases = [_Case(k, run, stored) for k in keys]
    flips = {}
    t0 = time.time()
    for l in range(g.n_layers):
        Wl = _layer_weights(view, g, l)
        for case in cases:
            rep = _layer_step(case, l, Wl)
            for k, v in rep.items():
                if isinstance(v, dict) and "flips" in v:
                    f = flips.setdefault((case.key, k), [0, 0])
                    f[0] += v["flips"]
                    f[1] += v["elements"]
            worst = max((v.get("max_ratio_to_bound", 0) for v in rep.values() if isinstance(v, dict)), default=0)
            print(f"{case.key} layer {l}: ok ({len(case.sample_rows(l))} rows; flip fractions "
                  + ", ".join(f"{k} {v['flip_fraction']:.4f}" for k, v in rep.items()
                              if isinstance(v, dict) and "flip_fraction" in v)
                  + f"; residual error / bound max {worst:.3g}) [{time.time() - t0:.0f} s]", flush=True)
        del Wl
    for case in cases:
        rep = _final_and_head(case, view)
        print(case.key, rep, flush=True)
    print("rounding flips over all layers:", {f"{k[0]}.{k[1]}": round(v[0] / max(v[1], 1), 5)
                                               for k, v in sorted(flips.items())}, flush=True)


def test_every_layer_stagewise_dream7b():
    """c4: Dream-7B geometry (GQA 28/4, q/k/v biases), B4 x 768 tokens, all 28 layers."""
    _run_geometry(["c4"])


def test_every_layer_stagewise_llada8b():
    """c2 (B1 x 384), c3 (B1 x 1280) and c5 (B8 x 64 after a 1216-key cached prefix): LLaDA-8B
    geometry, all 32 layers."""
    _run_geometry(["c2", "c3", "c5"])


# Ragged shapes at the same bounds: d_model 208 and d_ffn 400 are not multiples of the 64-deep stages
# (every GEMM runs its K-tail variant), 3 x 37 tokens, 13 / 208 / 800 / 256 weight rows and a 1000-id
# vocabulary do not fill their tiles (rows outside an operand are clamped), H * dh = 256 != d_model,
# GQA 4/2 with q/k/v biases, and a 13-token cached prefix (5 carried keys in front of the fresh ones).
_ODD = synth.Workload("odd_shapes", dataclasses.replace(synth.WORKLOADS["c1s"].geom, name="odd-shapes", n_layers=2,
                                                        n_heads=4, n_kv_heads=2, head_dim=64, d_model=208, d_ffn=400,
                                                        vocab=1000, mask_id=999, qkv_bias=True, weight_dtype="bf16",
                                                        rope_base=1e6),
                      batch=3, prompt_len=0, gen_len=37, window=16, p=0, draft=(20, 37), tau_commit=0.7,
                      tau_draft=0.98, kv_prefix=13, kv_seed=5)


def test_every_layer_stagewise_ragged_shapes():
    """Both layers of a small GQA + bias geometry whose every dimension leaves partial tiles and K tails."""
    stored = synth.make_weights(_ODD.geom)
    _run_geometry([_ODD], stored, runner_for(_ODD, stored))


# ---------------------------------------------------------------- LM head on its production plans

_HEAD = {
    "llada": dataclasses.replace(synth.LLADA8B, name="llada-head", n_layers=1),
    "dream": dataclasses.replace(synth.DREAM7B, name="dream-head", n_layers=1),
}
_head_cache = {}


@pytest.mark.parametrize("geom,n", [("llada", 384), ("llada", 512), ("llada", 1280), ("dream", 3072)])
def test_lm_head_production_plans_exact_bar(geom, n):
    """dcl_score_hidden at the token counts of the workloads, whose tuned plans have every wave own a whole
    128-id vocabulary tile (the wave-owned branch of the fused epilogue): conf within 1e-3, lse within 2e-2,
    ids exact except near-ties, entropy within the per-row bar, on the LLaDA-8B and Dream-7B vocabularies."""
    import torch
    import paper_2607_20467_amd as dcl
    g = _HEAD[geom]
    plan = dcl.dcl_debug_gemm_plan(g.vocab, n, g.d_model, lm_head=True)
    print(f"case head {geom} n={n} plan {plan}", flush=True)
    assert plan["bw"] // plan["ww"] == 128, f"plan {plan} does not give each wave a whole vocabulary tile"
    if geom not in _head_cache:
        _head_cache.clear()
        torch.cuda.empty_cache()
        stored = synth.make_weights(g)
        w = dataclasses.replace(synth.WORKLOADS["c2"], geom=g)
        _head_cache[geom] = (stored, runner_for(w, stored))
    stored, run = _head_cache[geom]
    h = synth.normal_bf16(78, n, 1.0, (n, g.d_model))
    st = stats_to_np(run.score_hidden(torch.from_numpy(h.view(np.int16)).cuda()))
    rng = np.random.default_rng([n, 7])
    pick = np.sort(rng.choice(n, min(HEAD_ROWS, n), replace=False))
    lg = oracle.lm_logits(WeightView(stored), synth.bf16_bits_to_f32(h[pick]).astype(np.float64))
    t1, t2, c, p2, lse = oracle.row_stats(lg)
    ent = oracle.row_entropy(lg)
    ref = {"top1": t1[None], "top2": t2[None], "conf": c[None], "p2": p2[None], "lse": lse[None], "entropy": ent[None]}
    gpu = {k: v[pick][None] for k, v in st.items()}
    P = np.exp(lg - lse[:, None])
    sd = np.sqrt(np.maximum((P * lg ** 2).sum(1) - (P * lg).sum(1) ** 2, 0.0))
    rep = compare_stats(gpu, ref, what=f"score_hidden[{geom}, n={n}]", entropy_tol=(LOGIT_TOL * np.maximum(sd, 1.0))[None])
    assert rep["meets_exact_input_bar"]
    np.testing.assert_allclose(st["p2"][pick], p2, atol=CONF_TOL)
    ok = (np.log(c) - np.log(p2) >= TIE_GAP) & (st["top1"][pick] == t1)
    np.testing.assert_array_equal(st["top2"][pick][ok], t2[ok])
