"""dcl_denoise_step_noalloc (the step with its workspace in the library's static scratch, for callers
that cannot allocate) against dcl_denoise_step with a caller workspace: the same kernels on the same
inputs, so the statistics must be identical bit for bit. Two calls in a row, the second on a smaller
input, check that the shared scratch carries nothing from one call into the next. The refusal of a step
whose workspace exceeds the scratch is a host-side check, tested without a GPU in test_abi.py (no GPU
test hands the library addresses that only that check keeps from being used)."""
import dataclasses

import numpy as np
import pytest

import synth

from helpers import runner_for, stats_to_np, to_dev

pytestmark = pytest.mark.gpu


def test_noalloc_step_matches_workspace_step():
    import paper_2607_20467_amd as dcl
    base = synth.WORKLOADS["c1s"]
    small = dataclasses.replace(base, batch=1, prompt_len=20, gen_len=44, window=16, p=20, draft=(36, 44))
    stored = synth.make_weights(base.geom)
    run = runner_for(base, stored)
    for w in (base, small):
        tok, p = synth.initial_state(w)
        B, S = tok.shape
        print(f"case noalloc B={B} S={S}", flush=True)
        t_dev, p_dev = to_dev(tok), to_dev(p)
        ref = stats_to_np(run.step(t_dev, p_dev, w.gen_end))
        got = run.new_stats(B, S)
        for v in got.values():
            v.fill_(7)                       # every entry must be written by the call
        dcl.dcl_denoise_step_noalloc(run.model, t_dev, B, S, p_dev, w.gen_end, None, 0, got)
        got = stats_to_np(got)
        for k in ref:
            np.testing.assert_array_equal(got[k], ref[k], err_msg=f"{k} differs at B={B} S={S}")
        assert (ref["conf"] >= 0).sum() > 0

