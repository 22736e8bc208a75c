"""Degenerate inputs of a whole step on the GPU, against the oracle:
* every sequence finished (p = gen_end): no row is scored, every statistic is the sentinel, and the
  selection changes nothing;
* a batch mixing finished and active sequences (one with a single uncommitted position);
* very short sequences: 8 tokens (one 8-key chunk, a single attention tile whose second key group
  is empty), 5 tokens (a one-token generation region, S not a multiple of 8), 2 tokens (one
  prompt token and one masked position) and a single masked token (one key, no prompt);
* a step whose selection finishes the sequence.
Statistics are compared within the whole-step tolerance (helpers.py), selections bit-exactly on
the GPU's own statistics."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from oracle.numerics import WeightView

from helpers import compare_stats, derived_tolerance, runner_for, stats_to_np, to_dev

pytestmark = pytest.mark.gpu

_C1 = synth.WORKLOADS["c1"]
_cache = {}


def _setup():
    if "c1" not in _cache:
        stored = synth.make_weights(_C1.geom)
        _cache["c1"] = (stored, WeightView(stored), runner_for(_C1, stored))
    return _cache["c1"]


def _workload(name, **kw):
    return dataclasses.replace(_C1, key=name, **kw)


def _step_and_select(w, tok, p):
    """GPU step + selection; returns (stats, tokens, p, K_raw, K_eff) as numpy."""
    import torch
    import paper_2607_20467_amd as dcl
    _, _, run = _setup()
    B, S = tok.shape
    t_dev, p_dev = to_dev(tok), to_dev(p)
    st = run.step(t_dev, p_dev, w.gen_end)
    kr = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    ke = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    stats = stats_to_np(st)
    dcl.dcl_select_contiguous(t_dev, B, S, p_dev, w.gen_end, w.window, w.tau_commit, w.tau_draft, w.geom.mask_id,
                              st, kr, ke)
    torch.cuda.synchronize()
    return stats, t_dev.cpu().numpy(), p_dev.cpu().numpy(), kr.cpu().numpy(), ke.cpu().numpy()


def _check(w, tok, p, what):
    _, W, _ = _setup()
    print(f"case {what}: B={tok.shape[0]} S={tok.shape[1]} p={p.tolist()} gen_end={w.gen_end}", flush=True)
    ref = oracle.step(w.geom, W, tok, p, w.gen_end)
    stats, t_gpu, p_gpu, kr, ke = _step_and_select(w, tok, p)
    if (ref["conf"] >= 0).any():
        ct, lt = derived_tolerance(w.geom, W, tok, p, w.gen_end, ref)
        compare_stats(stats, ref, w.tau_commit, w.tau_draft, what=what, conf_tol=ct, logit_tol=lt)
    else:
        np.testing.assert_array_equal(stats["conf"] >= 0, False)
        np.testing.assert_array_equal(stats["top1"], -1)
        np.testing.assert_array_equal(stats["conf"], -1.0)
    x_ref, p_ref, kr_ref, ke_ref = oracle.select_contiguous(
        tok, p, w.gen_end, w.window, w.tau_commit, w.tau_draft, w.geom.mask_id, stats["top1"],
        stats["conf"].astype(np.float64))
    np.testing.assert_array_equal(t_gpu, x_ref, err_msg=f"{what}: tokens")
    np.testing.assert_array_equal(p_gpu, p_ref, err_msg=f"{what}: p")
    np.testing.assert_array_equal(kr, kr_ref, err_msg=f"{what}: K_raw")
    np.testing.assert_array_equal(ke, ke_ref, err_msg=f"{what}: K_eff")
    return stats, t_gpu, p_gpu


def test_finished_sequences_score_nothing():
    w = _workload("finished", batch=2)
    tok, p = synth.initial_state(w)
    p[:] = w.gen_end
    stats, t_gpu, p_gpu = _check(w, tok, p, "finished")
    np.testing.assert_array_equal(t_gpu, tok)
    np.testing.assert_array_equal(p_gpu, p)


def test_mixed_finished_and_active():
    w = _workload("mixed", batch=3)
    tok, p = synth.initial_state(w)
    p[0] = w.gen_end                  # finished
    p[2] = w.gen_end - 1              # one uncommitted position left
    tok[2, : w.gen_end - 1] = np.where(tok[2, : w.gen_end - 1] == w.geom.mask_id, 7, tok[2, : w.gen_end - 1])
    _, t_gpu, p_gpu = _check(w, tok, p, "mixed")
    assert p_gpu[0] == w.gen_end and p_gpu[2] == w.gen_end   # the last position is always committed
    assert (t_gpu[2] != w.geom.mask_id).all()


@pytest.mark.parametrize("prompt_len,gen_len,window", [(4, 4, 4), (4, 1, 1), (1, 7, 3), (1, 1, 1), (0, 1, 1)])
def test_short_sequences(prompt_len, gen_len, window):
    w = _workload(f"short_{prompt_len}_{gen_len}", batch=2, prompt_len=prompt_len, gen_len=gen_len,
                  window=window, p=prompt_len, draft=(0, 0))
    tok, p = synth.initial_state(w)
    _check(w, tok, p, f"short S={w.seq}")
