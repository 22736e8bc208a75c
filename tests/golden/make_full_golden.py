"""Write the expected step statistics of the full-size workloads (c2-c5) with the float64 oracle.

Calls only ``oracle`` and ``synth``. For every workload it stores, per scored row, the oracle's
top1 / top2 / conf / p2 / lse, the drift of the same definition evaluated in float32 (which sizes
the whole-step tolerance), the oracle's selection on its own statistics, and checksums of a few
weight tensors so a machine that regenerates different weights is detected.

    python tests/golden/make_full_golden.py [--out DIR] [c1 c2 c3 c4 c5]
(c1: the draft placeholders of the tiny workload, c1_drafts.json)
(tens of minutes on 8 cores; DIR defaults to this directory)
"""
import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
import synth  # noqa: E402
from oracle.numerics import WeightView  # noqa: E402

CHECK_TENSORS = ("embed", "l0.wq", "l0.wd", "lm_head")


def checksums(stored):
    return {n: hashlib.sha256(np.ascontiguousarray(stored[n]).tobytes()).hexdigest()[:16] for n in CHECK_TENSORS}


OUT = HERE


def run(key, stored):
    w = synth.WORKLOADS[key]
    g = w.geom
    tok, p = synth.initial_state(w)
    kv = None
    if w.kv_prefix:
        caches = [synth.kv_cache_layer(w, l) for l in range(g.n_layers)]

        def kv(b, l):
            k, v = caches[l]
            return synth.bf16_bits_to_f32(k[b]), synth.bf16_bits_to_f32(v[b])
        kv.prefix = w.kv_prefix
    W = WeightView(stored)

    def per_sequence(**kw):
        """oracle.step one sequence at a time (the same result; a progress line after each)."""
        parts = []
        for b in range(tok.shape[0]):
            kvb = None
            if kv is not None:
                kvb = lambda bb, l, b=b: kv(b, l)
                kvb.prefix = kv.prefix
            parts.append(oracle.step(g, W, tok[b:b + 1], p[b:b + 1], w.gen_end, kv=kvb, **kw))
            print(f"  {key} sequence {b} ({kw.get('dtype', np.float64).__name__}) done", flush=True)
        return {k: np.concatenate([q[k] for q in parts]) for k in parts[0]}

    t0 = time.time()
    ref = per_sequence()
    t1 = time.time()
    f32 = per_sequence(dtype=np.float32)
    t2 = time.time()
    m = ref["conf"] >= 0
    rows = np.nonzero(m.reshape(-1))[0]
    x, pn, kr, ke = oracle.select_contiguous(tok, p, w.gen_end, w.window, w.tau_commit, w.tau_draft, g.mask_id,
                                             ref["top1"], ref["conf"])
    # the same selection on the float32 evaluation's statistics: how often a float32 implementation of the
    # definition alone already lands on another K
    _, _, kr32, _ = oracle.select_contiguous(tok, p, w.gen_end, w.window, w.tau_commit, w.tau_draft, g.mask_id,
                                             f32["top1"], f32["conf"].astype(np.float64))
    out = dict(tokens=tok, p=p, rows=rows.astype(np.int64),
               top1=ref["top1"].reshape(-1)[rows], top2=ref["top2"].reshape(-1)[rows],
               conf=ref["conf"].reshape(-1)[rows], p2=ref["p2"].reshape(-1)[rows], lse=ref["lse"].reshape(-1)[rows],
               drift_conf=np.float64(np.abs(f32["conf"][m] - ref["conf"][m]).max()),
               drift_lse=np.float64(np.abs(f32["lse"][m] - ref["lse"][m]).max()),
               f32_top1_flips=np.int64((f32["top1"][m] != ref["top1"][m]).sum()),
               f32_conf=f32["conf"].reshape(-1)[rows], f32_lse=f32["lse"].reshape(-1)[rows],
               f32_top1=f32["top1"].reshape(-1)[rows],
               sel_tokens=x, sel_p=pn, sel_k_raw=kr, sel_k_eff=ke, f32_sel_k_raw=kr32,
               checksum_names=np.array(CHECK_TENSORS), checksum_values=np.array([checksums(stored)[n] for n in CHECK_TENSORS]),
               oracle_seconds=np.float64(t1 - t0))
    np.savez_compressed(os.path.join(OUT, f"full_{key}.npz"), **out)
    print(f"{key}: {len(rows)} scored rows, oracle {t1 - t0:.0f} s, float32 evaluation {t2 - t1:.0f} s, "
          f"drift conf {out['drift_conf']:.3g} lse {out['drift_lse']:.3g}, K_eff {ke.tolist()}, "
          f"K of the float32 evaluation {kr32.tolist()}", flush=True)


def make_drafts(key):
    """Draft placeholders of a workload whose drafts are the previous step's top-1 predictions: the top-1 of
    a warm-up step on the same prompt with the whole generation region masked (p at the window start),
    over the draft region. Written to {key}_drafts.json."""
    import json
    w = synth.WORKLOADS[key]
    g = w.geom
    prompt = synth.prompts(w)
    B = prompt.shape[0]
    x = np.full((B, w.seq), g.mask_id, np.int64)
    x[:, :w.prompt_len] = prompt
    p = np.full(B, w.p, np.int64)
    st = oracle.step(g, WeightView(synth.make_weights(g)), x, p, w.gen_end)
    lo, hi = w.draft
    rec = {"_source": "top-1 of a float64 oracle step on the prompt followed by mask ids (tests/golden/"
                      "make_full_golden.py): the previous step's predictions that the workload places in its "
                      "draft region", "workload": key, "geometry": g.name, "draft_region": [lo, hi],
           "drafts": st["top1"][:, lo:hi].tolist(), "confidences": st["conf"][:, lo:hi].round(6).tolist()}
    with open(os.path.join(OUT, f"{key}_drafts.json"), "w") as f:
        json.dump(rec, f, indent=1)
    print(f"{key}: drafts {rec['drafts']}", flush=True)


def main(keys):
    cache = {}
    for key in keys:
        if key == "c1":
            make_drafts(key)
            continue
        g = synth.WORKLOADS[key].geom
        if g.name not in cache:
            cache.clear()
            t = time.time()
            cache[g.name] = synth.make_weights(g)
            print(f"generated {g.name} in {time.time() - t:.0f} s", flush=True)
        run(key, cache[g.name])


if __name__ == "__main__":
    args = sys.argv[1:]
    if args[:1] == ["--out"]:
        OUT = args[1]
        os.makedirs(OUT, exist_ok=True)
        args = args[2:]
    main(args or ["c2", "c3", "c5", "c4"])
