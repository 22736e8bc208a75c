"""dcl_generate (Algorithm 1 on the device, iterations replayed from a captured HIP graph) against
the eager loop of dcl_denoise_step + dcl_select_contiguous on the same state.

The eager loop is itself checked against the float64 oracle at every iteration
(test_gpu_step.py::test_full_loop_matches_oracle_every_iteration); here every replay of the graph
must reproduce it bit for bit: tokens, p, K_raw, K_eff after every iteration count, with the
program's own eager work and host synchronisations between the replays."""
import numpy as np
import pytest

import synth

from helpers import runner_for, to_dev

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS
_cache = {}


def _setup(key, gen_len=48, batch=None):
    if key not in _cache:
        w = W[key]
        stored = synth.make_weights(w.geom)
        _cache[key] = (w, runner_for(w, stored))
    w, run = _cache[key]
    prompt = synth.prompts(w)
    if batch is not None:
        prompt = prompt[:batch]
    N = prompt.shape[1]
    x = np.concatenate([prompt, np.full((prompt.shape[0], gen_len), w.geom.mask_id)], 1).astype(np.int32)
    p = np.full(prompt.shape[0], N, np.int32)
    return w, run, x, p


def _eager(run, w, x0, p0, L, tc, td, n_iter, score_flags=0, select_flags=0, kv=None, block_origin=0, block_len=0):
    """States after each of n_iter eager iterations (device-resident, synchronised between them)."""
    import torch
    import paper_2607_20467_amd as dcl
    from oracle.select import block_end
    B, S = x0.shape
    tok, p = to_dev(x0), to_dev(p0)
    # Algorithm 1's loop-top remask of the first window (the initial masks already cover it)
    xs = tok.cpu().numpy()
    for b in range(B):
        xs[b, p0[b]:min(p0[b] + L, block_end(int(p0[b]), S, block_origin, block_len))] = w.geom.mask_id
    tok.copy_(to_dev(xs))
    st = run.new_stats(B, S)
    kr = torch.zeros(B, dtype=torch.int32, device="cuda")
    ke = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = []
    for _ in range(n_iter):
        run.step(tok, p, S, stats=st, flags=score_flags, kv=kv)
        dcl.dcl_select_contiguous(tok, B, S, p, S, L, tc, td, w.geom.mask_id, st, kr, ke, select_flags,
                                  block_origin=block_origin, block_len=block_len)
        torch.cuda.synchronize()
        out.append((tok.cpu().numpy(), p.cpu().numpy(), kr.cpu().numpy(), ke.cpu().numpy()))
    return out


def _generate(run, w, x0, p0, L, tc, td, max_steps, check_every=1, score_flags=0, select_flags=0, hist=None,
              kv=None, block_origin=0, block_len=0):
    import torch
    import paper_2607_20467_amd as dcl
    B, S = x0.shape
    tok, p = to_dev(x0), to_dev(p0)
    st = run.new_stats(B, S)
    kr = torch.zeros(B, dtype=torch.int32, device="cuda")
    ke = torch.zeros(B, dtype=torch.int32, device="cuda")
    ws, n = run.workspace(B, S, 0 if kv is None else kv[2])
    steps = dcl.dcl_generate(run.model, tok, B, S, p, S, kv, score_flags, L, tc, td, select_flags, max_steps,
                             check_every, st, kr, ke, hist, ws, n, block_origin=block_origin, block_len=block_len)
    torch.cuda.synchronize()
    return steps, tok.cpu().numpy(), p.cpu().numpy(), kr.cpu().numpy(), ke.cpu().numpy()


def test_every_replay_matches_the_eager_loop():
    w, run, x0, p0 = _setup("c1s")
    L, tc, td = 16, 0.7, 0.9
    S = x0.shape[1]
    ref = _eager(run, w, x0, p0, L, tc, td, 48)
    n_done = next(i + 1 for i, (_, p, _, _) in enumerate(ref) if (p >= S).all())
    print("eager loop finished in", n_done, "iterations", flush=True)
    for k in range(1, n_done + 1):
        steps, tok, p, kr, ke = _generate(run, w, x0, p0, L, tc, td, max_steps=k)
        assert steps == k
        rt, rp, rkr, rke = ref[k - 1]
        np.testing.assert_array_equal(tok, rt, err_msg=f"tokens after {k} iterations")
        np.testing.assert_array_equal(p, rp, err_msg=f"p after {k} iterations")
        np.testing.assert_array_equal(kr, rkr, err_msg=f"K_raw after {k} iterations")
        np.testing.assert_array_equal(ke, rke, err_msg=f"K_eff after {k} iterations")
    # run to completion: stops at the first iteration where every p reached gen_end
    steps, tok, p, _, _ = _generate(run, w, x0, p0, L, tc, td, max_steps=1000)
    assert steps == n_done and (p == S).all()
    np.testing.assert_array_equal(tok, ref[n_done - 1][0])


def test_check_every_and_histogram():
    import torch
    w, run, x0, p0 = _setup("c1s")
    L, tc, td = 16, 0.6, 0.95
    S = x0.shape[1]
    ref = _eager(run, w, x0, p0, L, tc, td, 48)
    n_done = next(i + 1 for i, (_, p, _, _) in enumerate(ref) if (p >= S).all())
    hist = torch.zeros(L + 1, dtype=torch.int32, device="cuda")
    steps, tok, p, _, _ = _generate(run, w, x0, p0, L, tc, td, max_steps=1000, check_every=5, hist=hist)
    # completion is seen at the next multiple of 5; the extra iterations change nothing
    assert steps == -(-n_done // 5) * 5
    np.testing.assert_array_equal(tok, ref[n_done - 1][0])
    np.testing.assert_array_equal(p, ref[n_done - 1][1])
    # histogram: one count per (sequence, iteration) while the sequence was unfinished
    want = np.zeros(L + 1, np.int64)
    p_prev = p0
    for _, pk, _, kek in ref[:n_done]:
        for b in range(len(p_prev)):
            if p_prev[b] < S:
                want[kek[b]] += 1
        p_prev = pk
    np.testing.assert_array_equal(hist.cpu().numpy(), want)


def test_profiled_generate_runs_eagerly_and_agrees():
    import paper_2607_20467_amd as dcl
    w, run, x0, p0 = _setup("c1s")
    L, tc, td = 16, 0.7, 0.9
    a = _generate(run, w, x0, p0, L, tc, td, max_steps=1000)
    dcl.dcl_profile_enable(True)
    try:
        b = _generate(run, w, x0, p0, L, tc, td, max_steps=1000)
        prof = dcl.dcl_profile_read()
    finally:
        dcl.dcl_profile_enable(False)
    assert a[0] == b[0]
    for u, v in zip(a[1:], b[1:]):
        np.testing.assert_array_equal(u, v)
    assert prof["select"][0] == b[0]  # one select launch per iteration, each with its event pair


def test_score_all_mode_replays_match():
    import paper_2607_20467_amd as dcl
    w, run, x0, p0 = _setup("c1s")
    L, tc, td = 16, 0.7, 0.9
    sf, sel = dcl.DCL_SCORE_ALL_UNCOMMITTED, dcl.DCL_SEL_SCORE_ALL
    ref = _eager(run, w, x0, p0, L, tc, td, 6, score_flags=sf, select_flags=sel)
    steps, tok, p, kr, ke = _generate(run, w, x0, p0, L, tc, td, max_steps=6, score_flags=sf, select_flags=sel)
    assert steps == 6
    np.testing.assert_array_equal(tok, ref[-1][0])
    np.testing.assert_array_equal(p, ref[-1][1])


def test_cached_prefix_replays_match_the_eager_loop():
    """The prompt's keys/values go into a cache once (dcl_kv_append); the loop then forwards only the
    generation region, which attends to [cached prompt || itself] (the prefix-KV decode mode)."""
    import torch
    w, run, x0, p0 = _setup("c1s")
    g = w.geom
    B, N = x0.shape[0], int(p0[0])
    assert N % 8 == 0
    ks = [torch.zeros((B, g.n_kv_heads, N, g.head_dim), dtype=torch.int16, device="cuda") for _ in range(g.n_layers)]
    vs = [torch.zeros((B, g.n_kv_heads, g.head_dim, N), dtype=torch.int16, device="cuda") for _ in range(g.n_layers)]
    run.kv_append(to_dev(np.ascontiguousarray(x0[:, :N])), (ks, vs, 0, N))
    kv = (ks, vs, N, N)
    x = np.ascontiguousarray(x0[:, N:])
    p = np.zeros(B, np.int32)
    S = x.shape[1]
    L, tc, td = 16, 0.7, 0.9
    ref = _eager(run, w, x, p, L, tc, td, 48, kv=kv)
    n_done = next(i + 1 for i, (_, pk, _, _) in enumerate(ref) if (pk >= S).all())
    print("cached-prefix eager loop finished in", n_done, "iterations", flush=True)
    for k in sorted({1, 2, 3, n_done}):
        steps, tok, pk, kr, ke = _generate(run, w, x, p, L, tc, td, max_steps=k, kv=kv)
        assert steps == k
        rt, rp, rkr, rke = ref[k - 1]
        np.testing.assert_array_equal(tok, rt, err_msg=f"tokens after {k} iterations")
        np.testing.assert_array_equal(pk, rp, err_msg=f"p after {k} iterations")
        np.testing.assert_array_equal(kr, rkr, err_msg=f"K_raw after {k} iterations")
        np.testing.assert_array_equal(ke, rke, err_msg=f"K_eff after {k} iterations")
    # the cache is read, never written, by the loop
    ks2 = [k.clone() for k in ks]
    _generate(run, w, x, p, L, tc, td, max_steps=1000, kv=kv)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(ks, ks2))


def test_blocked_generation_replays_the_eager_loop():
    """dcl_generate with semi-autoregressive blocks (block origin at the prompt end, blocks of 8, window 16)
    reproduces the eager blocked loop bit for bit and finishes at the same iteration."""
    w, run, x0, p0 = _setup("c1s")
    L, tc, td, BL = 16, 0.6, 0.9, 8
    N, S = int(p0[0]), x0.shape[1]
    ref = _eager(run, w, x0, p0, L, tc, td, 48, block_origin=N, block_len=BL)
    n_done = next(i + 1 for i, (_, p, _, _) in enumerate(ref) if (p >= S).all())
    for k in (1, 2, n_done // 2, n_done):
        steps, tok, p, kr, ke = _generate(run, w, x0, p0, L, tc, td, max_steps=k, block_origin=N, block_len=BL)
        assert steps == k
        for name, g, r in zip(("tokens", "p", "K_raw", "K_eff"), (tok, p, kr, ke), ref[k - 1]):
            np.testing.assert_array_equal(g, r, err_msg=f"{name} after {k} blocked iterations")
    # every block end is reached: p never jumps over one
    for b in range(x0.shape[0]):
        visited = {int(r[1][b]) for r in ref[:n_done]}
        assert {N + BL * j for j in range(1, (S - N) // BL + 1)} <= visited


@pytest.mark.parametrize("key,block_len", [("c1", 0), ("c1", 16), ("c1s", 0), ("c1s", 16)])
def test_whole_trajectory_against_oracle_generate(tiny_weights, key, block_len):
    """Algorithm 1 end to end on the GPU against oracle.generate from the same prompt (64 generated tokens,
    window 16, tau_c 0.7, tau_d 0.98; blocks of 16 or none), compared iteration by iteration. Either the
    trajectories are equal, or the first iteration where they part is reported with what decided it: an
    acceptance length set by a window row whose oracle confidence lies within that state's derived
    confidence tolerance of tau_c, a committed id at a near-tie row, or a draft decision at a row within the
    tolerance of tau_d. The GPU and the oracle start that iteration from the same state."""
    import oracle
    from helpers import derived_tolerance
    w, stored, Wv = tiny_weights(key)
    M, L, tc, td = 64, 16, 0.7, 0.98
    _, run, x0, p0 = _setup(key, gen_len=M)
    N = int(p0[0])
    S = x0.shape[1]
    prompt = x0[:, :N]
    trace = []
    x_or, steps_or = oracle.generate(w.geom, Wv, prompt, M, L, tc, td, trace=trace, block_len=block_len)
    gpu = _eager(run, w, x0, p0, L, tc, td, len(trace) + 8, block_origin=N, block_len=block_len)
    steps_gpu = next(i + 1 for i, (_, p, _, _) in enumerate(gpu) if (p >= S).all())
    prev_x = x0.copy()
    prev_p = p0.astype(np.int64)
    for it, ((gx, gp, gkr, gke), (ox, op, okr, oke)) in enumerate(zip(gpu, trace)):
        if np.array_equal(gx, ox) and np.array_equal(gp, op):
            prev_x, prev_p = ox, op
            continue
        ref = oracle.step(w.geom, Wv, prev_x, prev_p, S)
        ct, lt = derived_tolerance(w.geom, Wv, prev_x, prev_p, S, ref)
        gap = np.log(np.maximum(ref["conf"], 1e-300)) - np.log(np.maximum(ref["p2"], 1e-300))
        for b in range(x0.shape[0]):
            if gkr[b] != okr[b]:
                j = int(prev_p[b]) + min(int(gkr[b]), int(okr[b]))
                d = abs(ref["conf"][b, j] - tc)
                print(f"{key} blocks {block_len}: iteration {it + 1} of {steps_or}, seq {b}: K GPU {gkr[b]}, oracle "
                      f"{okr[b]}; deciding row {j}: oracle conf {ref['conf'][b, j]:.5f}, |c - tau_c| = {d:.5f} "
                      f"(state's confidence tolerance {ct:.5f})", flush=True)
                assert d <= ct
                continue
            for j in np.nonzero(gx[b] != ox[b])[0]:
                committed = prev_p[b] <= j < op[b]
                why = (f"top-1/top-2 logit gap {gap[b, j]:.4f} (tolerance {lt:.4f})" if committed else
                       f"draft row: |c - tau_d| = {abs(ref['conf'][b, j] - td):.5f}, gap {gap[b, j]:.4f}")
                print(f"{key} blocks {block_len}: iteration {it + 1} of {steps_or}, seq {b}: token at {j} differs, "
                      f"{why}", flush=True)
                assert gap[b, j] < lt or (not committed and abs(ref["conf"][b, j] - td) <= ct)
        break
    else:
        assert steps_gpu == steps_or and np.array_equal(gpu[steps_gpu - 1][0], x_or)
        print(f"{key} blocks {block_len}: the GPU trajectory equals the oracle's ({steps_or} iterations)", flush=True)
