"""A caller can capture dcl_denoise_step + dcl_select_contiguous into its own HIP graph (torch's
CUDAGraph on a side stream): no call allocates, synchronises or records a memset. Every replay,
with the program's own eager work and synchronisations between replays, reproduces the eager
call bit for bit (statistics, tokens, p, K). Two steps in flight on two streams, each with its own
workspace, do not interfere."""
import numpy as np
import pytest

import synth

from helpers import runner_for, to_dev
from test_gpu_step import CASES

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("key", ["c1s", "ragged", "many_heads"])
def test_captured_step_replays_match_eager(key):
    import torch
    import paper_2607_20467_amd as dcl
    w = CASES[key]
    g = w.geom
    run = runner_for(w, synth.make_weights(g))
    tok_h, p_h = synth.initial_state(w)
    B, S = tok_h.shape
    tok0, p0 = to_dev(tok_h), to_dev(p_h)
    tok, p = tok0.clone(), p0.clone()
    stats = run.new_stats(B, S)
    ws, n = run.workspace(B, S)
    kr = torch.zeros(B, dtype=torch.int32, device="cuda")
    ke = torch.zeros(B, dtype=torch.int32, device="cuda")

    def one_step(stream):
        tok.copy_(tok0, non_blocking=True)
        p.copy_(p0, non_blocking=True)
        dcl.dcl_denoise_step(run.model, tok, B, S, p, w.gen_end, None, 0, stats, ws, n, stream)
        dcl.dcl_select_contiguous(tok, B, S, p, w.gen_end, w.window, w.tau_commit, w.tau_draft, g.mask_id, stats,
                                  kr, ke, 0, stream)

    def snapshot():
        torch.cuda.synchronize()
        out = {k: v.cpu().numpy().copy() for k, v in stats.items()}
        out.update(tokens=tok.cpu().numpy(), p=p.cpu().numpy(), k_raw=kr.cpu().numpy(), k_eff=ke.cpu().numpy())
        return out

    main = torch.cuda.current_stream()
    one_step(main)
    ref = snapshot()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(main)
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            one_step(side)
    torch.cuda.synchronize()
    for r in range(3):
        for v in stats.values():               # eager work between replays
            v.fill_(-3)
        kr.fill_(-3)
        tok.zero_()
        torch.cuda.synchronize()
        graph.replay()
        got = snapshot()
        for k in ref:
            np.testing.assert_array_equal(got[k], ref[k], err_msg=f"{key}: replay {r}, {k}")
    # an eager call after the replays still agrees
    one_step(main)
    got = snapshot()
    for k in ref:
        np.testing.assert_array_equal(got[k], ref[k], err_msg=f"{key}: eager after replays, {k}")


def test_two_streams_with_separate_workspaces():
    """Two steps of one model in flight at once on two streams, each with its own workspace and
    outputs, give the results of running them one after the other."""
    import torch
    import paper_2607_20467_amd as dcl
    w = CASES["c1s"]
    g = w.geom
    run = runner_for(w, synth.make_weights(g))
    tok_h, p_h = synth.initial_state(w)
    B, S = tok_h.shape
    tok_b = tok_h.copy()
    tok_b[:, w.p:w.p + 4] = 17                       # a different state for the second step
    p_b = p_h + 4
    n = dcl.dcl_workspace_bytes(run.model, B, S, 0)

    def launch(tok, p, stream):
        ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        st = run.new_stats(B, S)
        t, pp = to_dev(tok), to_dev(p)
        torch.cuda.synchronize()
        dcl.dcl_denoise_step(run.model, t, B, S, pp, w.gen_end, None, 0, st, ws, n, stream)
        return st, (ws, t, pp)      # every buffer the stream reads stays alive until it has finished

    ref_a = {k: v.cpu().numpy() for k, v in launch(tok_h, p_h, torch.cuda.current_stream())[0].items()}
    ref_b = {k: v.cpu().numpy() for k, v in launch(tok_b, p_b, torch.cuda.current_stream())[0].items()}
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for _ in range(3):
        st_a, keep_a = launch(tok_h, p_h, s1)
        st_b, keep_b = launch(tok_b, p_b, s2)
        torch.cuda.synchronize()
        for k in ref_a:
            np.testing.assert_array_equal(st_a[k].cpu().numpy(), ref_a[k], err_msg=f"stream 1: {k}")
            np.testing.assert_array_equal(st_b[k].cpu().numpy(), ref_b[k], err_msg=f"stream 2: {k}")
