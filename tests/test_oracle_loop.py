"""Pins for the full decode loop of Algorithm 1 (Appendix A), CPU."""
import json

import numpy as np

import oracle
import synth
from oracle.loop import generate, sequential_greedy


def _setup(tiny_weights, key="c1s"):
    w, stored, W = tiny_weights(key)
    return w, W, synth.prompts(w)


def test_loop_invariants(tiny_weights):
    """Committed tokens form a left-anchored run that only grows; history never changes; p strictly
    increases; the loop ends within M steps."""
    w, W, prompt = _setup(tiny_weights)
    M, L = 40, 8
    trace = []
    x, steps = generate(w.geom, W, prompt, M, L, 0.7, 0.98, trace=trace)
    N = prompt.shape[1]
    assert steps <= M
    prev_x = np.concatenate([prompt, np.full((prompt.shape[0], M), w.geom.mask_id)], 1)
    prev_p = np.full(prompt.shape[0], N)
    for xt, pt, kr, ke in trace:
        for b in range(prompt.shape[0]):
            if prev_p[b] < N + M:
                assert pt[b] > prev_p[b] and ke[b] >= 1 and ke[b] == max(kr[b], 1)
            np.testing.assert_array_equal(xt[b, :prev_p[b]], prev_x[b, :prev_p[b]])
        prev_x, prev_p = xt, pt
    np.testing.assert_array_equal(x[:, :N], prompt)
    assert (prev_p == N + M).all()


def test_loop_with_tau_one_is_sequential_greedy(tiny_weights):
    """tau_commit >= 1 accepts nothing, so K_eff = 1 every step; with drafts disabled (tau_draft > 1)
    Algorithm 1 reduces to chain-rule greedy decoding (Section 2.2, Eq. sequential_chain)."""
    w, W, prompt = _setup(tiny_weights)
    M, L = 12, 4
    x, steps = generate(w.geom, W, prompt, M, L, 1.0, 1.01)
    assert steps == M
    np.testing.assert_array_equal(x, sequential_greedy(w.geom, W, prompt, M))


def test_single_window_tau_zero_commits_one_forward_argmax(tiny_weights):
    """L = M and tau_commit = 0: the first iteration accepts the whole generation region, i.e. the
    top-1 of one forward over prompt + M masks."""
    w, W, prompt = _setup(tiny_weights)
    M = 16
    N = prompt.shape[1]
    x, steps = generate(w.geom, W, prompt, M, M, 0.0, 0.98)
    assert steps == 1
    x0 = np.concatenate([prompt, np.full((prompt.shape[0], M), w.geom.mask_id)], 1)
    st = oracle.step(w.geom, W, x0, np.full(prompt.shape[0], N), N + M)
    np.testing.assert_array_equal(x[:, N:], st["top1"][:, N:])


def test_checkpoint_resume(tiny_weights, tmp_path):
    """A step is a pure function of (weights, x, p, params): saving (x, p) mid-run and resuming gives
    the uninterrupted result."""
    w, W, prompt = _setup(tiny_weights)
    M, L = 32, 8
    trace = []
    full, _ = generate(w.geom, W, prompt, M, L, 0.7, 0.98, trace=trace)
    x3, p3 = trace[2][0], trace[2][1]
    ck = tmp_path / "state.json"
    ck.write_text(json.dumps({"x": x3.tolist(), "p": p3.tolist()}))
    st = json.loads(ck.read_text())
    x, p = np.array(st["x"]), np.array(st["p"])
    end = prompt.shape[1] + M
    while (p < end).any():
        s = oracle.step(w.geom, W, x, p, end)
        x, p, _, _ = oracle.select_contiguous(x, p, end, L, 0.7, 0.98, w.geom.mask_id, s["top1"], s["conf"])
    np.testing.assert_array_equal(x, full)


def test_drafts_written_and_later_invalidated(tiny_weights):
    """Drafts appear only at positions >= p + L and are re-masked once the window reaches them."""
    w, W, prompt = _setup(tiny_weights)
    M, L = 40, 8
    trace = []
    generate(w.geom, W, prompt, M, L, 0.7, 0.9, trace=trace)
    N = prompt.shape[1]
    mask = w.geom.mask_id
    saw_draft = False
    for xt, pt, _, _ in trace:
        for b in range(prompt.shape[0]):
            window = xt[b, pt[b]:min(pt[b] + L, N + M)]
            assert (window == mask).all()
            if (xt[b, pt[b] + L:] != mask).any():
                saw_draft = True
    assert saw_draft


# ---------------------------------------------------------------- semi-autoregressive blocks (reading R24)

def test_block_end_tiles_the_generation_region():
    from oracle.select import block_end
    assert [block_end(p, 100, 32, 16) for p in (32, 40, 47, 48, 95, 96, 99)] == [48, 48, 48, 64, 96, 100, 100]
    assert block_end(50, 100, 32, 0) == 100                      # no blocks: the generation end
    assert block_end(31, 100, 32, 16) == 32                      # before the origin: the origin


def test_one_block_covering_the_region_is_no_blocking(tiny_weights):
    w, W, prompt = _setup(tiny_weights)
    M, L = 24, 8
    a, sa = generate(w.geom, W, prompt, M, L, 0.7, 0.9)
    b, sb = generate(w.geom, W, prompt, M, L, 0.7, 0.9, block_len=M)
    np.testing.assert_array_equal(a, b)
    assert sa == sb


def test_blocks_of_one_token_are_sequential_greedy(tiny_weights):
    """Blocks of length 1 clip every window to one position: with drafts off each iteration commits the
    top-1 at p, i.e. chain-rule greedy decoding (Section 2.2), whatever tau_commit is."""
    w, W, prompt = _setup(tiny_weights)
    M = 10
    x, steps = generate(w.geom, W, prompt, M, 8, 0.0, 1.01, block_len=1)
    assert steps == M
    np.testing.assert_array_equal(x, sequential_greedy(w.geom, W, prompt, M))


def test_window_never_crosses_a_block_end(tiny_weights):
    """With blocks of 8 and a window of 16: each iteration commits inside the block holding p, p lands
    on every block end (no block is skipped), the re-masked window stops at the block end, and drafts
    past p + L are still written."""
    w, W, prompt = _setup(tiny_weights)
    M, L, BL = 32, 16, 8
    N = prompt.shape[1]
    trace = []
    generate(w.geom, W, prompt, M, L, 0.2, 0.5, trace=trace, block_len=BL)
    mask = w.geom.mask_id
    prev_p = np.full(prompt.shape[0], N)
    visited = [set([N]) for _ in range(prompt.shape[0])]
    saw_draft = False
    for xt, pt, kr, ke in trace:
        for b in range(prompt.shape[0]):
            if prev_p[b] >= N + M:
                continue
            be = N + BL * ((prev_p[b] - N) // BL + 1)
            assert pt[b] <= be                                   # the commit stayed in the block
            visited[b].add(int(pt[b]))
            nbe = min(N + M, N + BL * ((pt[b] - N) // BL + 1))
            assert (xt[b, pt[b]:nbe] == mask).all()
            if pt[b] + L < N + M and (xt[b, pt[b] + L:] != mask).any():
                saw_draft = True
        prev_p = pt
    for b in range(prompt.shape[0]):
        assert {N + k * BL for k in range(M // BL + 1)} <= visited[b]
    assert saw_draft
