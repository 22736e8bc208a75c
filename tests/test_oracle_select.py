"""Pins for the oracle's statistics and selection rules (CPU)."""
import itertools
import json
import os

import numpy as np
import pytest
import scipy.special

import oracle
from oracle.loop import noncontiguous_commit_set
from oracle.select import compute_k, scored_mask, select_contiguous

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "select_cases.json")


# ---------------------------------------------------------------- statistics (Section 2.1 / 2.2)

def test_row_stats_against_scipy_and_bruteforce():
    rng = np.random.default_rng(0)
    l = rng.standard_normal((50, 300)) * 4
    t1, t2, c, p2, lse = oracle.row_stats(l)
    P = scipy.special.softmax(l, axis=1)
    for r in range(50):                                 # brute-force scan
        best = max(range(300), key=lambda v: (l[r, v], -v))
        second = max((v for v in range(300) if v != best), key=lambda v: (l[r, v], -v))
        assert (t1[r], t2[r]) == (best, second)
        assert c[r] == pytest.approx(P[r].max(), rel=1e-12)
        assert p2[r] == pytest.approx(P[r, second], rel=1e-12)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(l, axis=1), rtol=1e-13)


def test_row_stats_special_cases():
    V = 1000
    t1, t2, c, p2, lse = oracle.row_stats(np.zeros((1, V)))       # uniform: conf = 1/V, ids 0 and 1
    assert (t1[0], t2[0]) == (0, 1) and c[0] == pytest.approx(1 / V) and p2[0] == pytest.approx(1 / V)
    assert lse[0] == pytest.approx(np.log(V))
    l = np.zeros((1, V)); l[0, 17] = l[0, 400] = 5.0             # tie: lower id wins, equal probabilities
    t1, t2, c, p2, _ = oracle.row_stats(l)
    assert (t1[0], t2[0]) == (17, 400) and c[0] == p2[0]
    l = np.zeros((1, V)); l[0, 999] = 1000.0                      # one-hot limit
    t1, t2, c, p2, _ = oracle.row_stats(l)
    assert t1[0] == 999 and t2[0] == 0 and c[0] == 1.0 and p2[0] < 1e-300


def test_row_stats_invariants():
    rng = np.random.default_rng(1)
    V = 4096
    l = rng.standard_normal((200, V)) * rng.uniform(0.1, 20, (200, 1))
    t1, t2, c, p2, _ = oracle.row_stats(l)
    assert (t1 != t2).all()
    assert (c >= 1 / V - 1e-15).all() and (c <= 1).all()
    assert (p2 <= c).all() and (p2 <= 1 - c + 1e-15).all()


# ---------------------------------------------------------------- DCV (Section 3.2, Eq. compute_k)

def test_golden_k_cases():
    cases = json.load(open(GOLDEN))["k_cases"]
    for case in cases:
        assert compute_k(np.array(case["conf"]), case["tau"]) == case["K"], case["why"]


@pytest.mark.parametrize("L", range(1, 13))
def test_compute_k_exhaustive(L):
    """K equals the index of the first failing entry (or L), for every pass/fail pattern of length L."""
    tau = 0.7
    for bits in itertools.product((0, 1), repeat=L):
        conf = np.where(np.array(bits) == 1, 0.9, 0.3)
        s = "".join(map(str, bits)) + "0"
        assert compute_k(conf, tau) == s.index("0")


def test_compute_k_thresholds_at_extremes():
    rng = np.random.default_rng(2)
    conf = rng.uniform(1e-6, 1, 64)
    assert compute_k(conf, 0.0) == 64          # tau = 0: every window entry is accepted
    assert compute_k(conf, 1.0) == 0           # tau >= 1: nothing is accepted (K_eff = 1)


# ---------------------------------------------------------------- commit / drafts / remask

@pytest.mark.parametrize("case", json.load(open(GOLDEN))["select_cases"], ids=lambda c: c["name"])
def test_golden_select_cases(case):
    tok = np.array([case["tokens"]])
    x, p, kr, ke = select_contiguous(tok, np.array([case["p"]]), case["gen_end"], case["L"],
                                     case["tau_commit"], case["tau_draft"], case["mask_id"],
                                     np.array([case["top1"]]), np.array([case["conf"]]),
                                     block_origin=case.get("block_origin", 0), block_len=case.get("block_len", 0))
    assert x[0].tolist() == case["expect_tokens"]
    assert (p[0], kr[0], ke[0]) == (case["expect_p"], case["expect_K_raw"], case["expect_K_eff"])


def _random_state(rng, B=6, S=80, mask=999):
    tok = rng.integers(0, 900, (B, S))
    p = rng.integers(5, S, B)
    for b in range(B):
        tok[b, p[b]:] = np.where(rng.random(S - p[b]) < 0.7, mask, tok[b, p[b]:])
    return tok, p


def test_select_rules_per_position():
    """Each output position obeys exactly one of: prompt/committed (unchanged), commit, draft, remask."""
    rng = np.random.default_rng(3)
    mask, S, L, end = 999, 80, 12, 80
    for trial in range(200):
        tok, p = _random_state(rng, S=S, mask=mask)
        sc = scored_mask(tok, p, end, mask)
        conf = np.where(sc, rng.uniform(0, 1, tok.shape), -1.0)
        top1 = np.where(sc, rng.integers(0, 900, tok.shape), -1)
        tc, td = rng.uniform(0.2, 0.9), rng.uniform(0.8, 1.0)
        x, pn, kr, ke = select_contiguous(tok, p, end, L, tc, td, mask, top1, conf)
        for b in range(tok.shape[0]):
            pb = p[b]
            Le = min(L, end - pb)
            first_fail = next((j for j in range(Le) if not conf[b, pb + j] > tc), Le)
            # reading R18: an unscored window start (no prediction at p) commits nothing
            want_ke = max(first_fail, 1) if top1[b, pb] >= 0 else first_fail
            assert kr[b] == first_fail and ke[b] == want_ke and pn[b] == pb + ke[b]
            assert (x[b] >= 0).all()                                                     # no sentinel committed
            np.testing.assert_array_equal(x[b, :pb], tok[b, :pb])                       # history immutable
            np.testing.assert_array_equal(x[b, pb:pn[b]], top1[b, pb:pn[b]])             # commit
            np.testing.assert_array_equal(x[b, pn[b]:min(pn[b] + L, end)], mask)         # remask
            for j in range(min(pn[b] + L, end), end):
                if j < pb + L:                                                           # old window
                    assert x[b, j] == tok[b, j]
                elif tok[b, j] == mask and conf[b, j] > td:
                    assert x[b, j] == top1[b, j]                                         # draft update
                else:
                    assert x[b, j] == tok[b, j]


def test_no_progress_guard_flag_and_score_all():
    tok = np.array([[1, 2, 9, 9, 9, 50, 9, 9]])
    top1 = np.array([[-1, -1, 30, 31, 32, 33, 34, 35]])
    conf = np.array([[-1, -1, 0.5, 0.99, 0.99, 0.995, 0.2, 0.99]])
    x, p, kr, ke = select_contiguous(tok, np.array([2]), 8, 3, 0.7, 0.98, 9, top1, conf,
                                     no_progress_guard=True)
    assert (kr[0], ke[0], p[0]) == (0, 0, 2)
    assert x[0].tolist() == [1, 2, 9, 9, 9, 50, 9, 35]            # nothing committed; drafts still update
    x, p, kr, ke = select_contiguous(tok, np.array([2]), 8, 3, 0.7, 0.98, 9, top1, conf, score_all=True)
    assert x[0].tolist() == [1, 2, 30, 9, 9, 9, 9, 35]             # window [3,6) re-masks position 5's redraft


def test_contiguous_commits_subset_of_threshold_commits():
    """For the same confidences, DCV's accepted window is a subset of Eq. threshold_pd's set."""
    rng = np.random.default_rng(4)
    for _ in range(500):
        conf = rng.uniform(0, 1, 40)
        tau = rng.uniform(0, 1)
        K = compute_k(conf[10:26], tau)
        assert set(range(10, 10 + K)) <= noncontiguous_commit_set(conf, 10, 26, tau)


# ---------------------------------------------------------------- selection variants

def test_row_stats_exclude_equals_vocabulary_without_that_id():
    """Mask-id suppression: the statistics are those of the softmax over V with the id deleted."""
    rng = np.random.default_rng(5)
    l = rng.standard_normal((40, 97)) * 3
    ex = 13
    l[:20, ex] = l[:20].max(axis=1) + 2.0          # the excluded id would be the argmax in half the rows
    t1, t2, c, p2, lse = oracle.row_stats(l, exclude=ex)
    keep = np.array([v for v in range(97) if v != ex])
    r1, r2, rc, rp2, rlse = oracle.row_stats(l[:, keep])
    np.testing.assert_array_equal(t1, keep[r1])
    np.testing.assert_array_equal(t2, keep[r2])
    np.testing.assert_allclose(c, rc, rtol=1e-14)
    np.testing.assert_allclose(p2, rp2, rtol=1e-14)
    np.testing.assert_allclose(lse, rlse, rtol=1e-14)
    assert not (t1 == ex).any() and not (t2 == ex).any()
    # without the flag the argmax of the first rows is the (unsuppressed) id
    assert (oracle.row_stats(l)[0][:20] == ex).all()


def _state(S, p, mask, filled=()):
    x = np.full((1, S), mask, np.int64)
    x[0, :p] = 7
    for j in filled:
        x[0, j] = 9
    return x, np.array([p])


def test_noncontiguous_rule_by_hand():
    mask, S, L = 99, 20, 6
    x, p = _state(S, 4, mask, filled=(6,))          # position 6 already holds a token
    conf = np.full((1, S), 0.2)
    conf[0, [4, 5, 7, 8]] = [0.95, 0.1, 0.9, 0.85]
    conf[0, 6] = -1.0                                # not scored (not masked)
    top1 = np.arange(S)[None] + 1000
    xn, pn, kr, ke = oracle.select_noncontiguous(x, p, S, L, 0.8, mask, top1, conf)
    # window [4, 10): masked rows 4, 5, 7, 8, 9; passing > 0.8: 4, 7, 8 (independent decisions)
    assert (kr[0], ke[0]) == (3, 3)
    assert [int(v) for v in xn[0, 4:10]] == [1004, mask, 9, 1007, 1008, mask]
    assert pn[0] == 5                                # first position still masked
    # nothing passes: the most confident masked row is committed (lowest position on ties)
    conf2 = np.full((1, S), 0.3)
    conf2[0, 6] = -1.0
    conf2[0, [7, 9]] = 0.5
    xn, pn, kr, ke = oracle.select_noncontiguous(x, p, S, L, 0.8, mask, top1, conf2)
    assert (kr[0], ke[0]) == (0, 1) and xn[0, 7] == 1007 and pn[0] == 4
    xn, pn, kr, ke = oracle.select_noncontiguous(x, p, S, L, 0.8, mask, top1, conf2, no_progress_guard=True)
    assert (kr[0], ke[0]) == (0, 0) and (xn == x).all() and pn[0] == 4


def test_noncontiguous_equals_contiguous_when_the_passing_set_is_a_prefix():
    """If the positions above the threshold form a leading run of the window (and every window row is
    masked), the independent rule commits exactly what Eq. compute_k commits, and both advance p to
    the end of that run (drafts off)."""
    rng = np.random.default_rng(9)
    mask, S, L, tau = 50, 40, 8, 0.7
    for trial in range(200):
        p0 = int(rng.integers(0, S - 1))
        x, p = _state(S, p0, mask)
        L_eff = min(L, S - p0)
        K = int(rng.integers(1, L_eff + 1))
        conf = rng.uniform(0.0, 0.7, (1, S))
        conf[0, p0:p0 + K] = rng.uniform(0.71, 1.0, K)
        top1 = rng.integers(0, 49, (1, S))
        a = oracle.select_noncontiguous(x, p, S, L, tau, mask, top1, conf)
        b = oracle.select_contiguous(x, p, S, L, tau, 2.0, mask, top1, conf)
        np.testing.assert_array_equal(a[0], b[0])
        np.testing.assert_array_equal(a[1], b[1])
        assert a[2][0] == b[2][0] == K


def test_contiguous_drafts_take_the_leading_chain():
    mask, S, L = 99, 30, 4
    x, p = _state(S, 2, mask, filled=(12,))         # an earlier draft at 12 (not masked, not scored)
    conf = np.full((1, S), 0.1)
    conf[0, 2:6] = 0.99                             # K = 4: p moves to 6 and [6, 10) is remasked afterwards
    conf[0, 12] = -1.0
    conf[0, [6, 7, 8, 9, 10, 11, 13, 14, 17, 18]] = 0.99   # chain from the old p + L = 6 breaks at 15
    top1 = np.arange(S)[None] + 500
    free = oracle.select_contiguous(x, p, S, L, 0.9, 0.95, mask, top1, conf)
    chain = oracle.select_contiguous(x, p, S, L, 0.9, 0.95, mask, top1, conf, contiguous_drafts=True)
    drafted = lambda r: [j for j in range(10, S) if r[0][0, j] not in (mask, 9)]
    assert free[1][0] == chain[1][0] == 6
    assert drafted(free) == [10, 11, 13, 14, 17, 18]
    assert drafted(chain) == [10, 11, 13, 14]
    # when every eligible draft row passes, the two rules agree
    conf[0, [15, 16] + list(range(19, S))] = 0.99
    a = oracle.select_contiguous(x, p, S, L, 0.9, 0.95, mask, top1, conf)
    b = oracle.select_contiguous(x, p, S, L, 0.9, 0.95, mask, top1, conf, contiguous_drafts=True)
    np.testing.assert_array_equal(a[0], b[0])


def test_row_entropy_against_scipy_and_extremes():
    import scipy.stats
    rng = np.random.default_rng(3)
    l = rng.standard_normal((30, 200)) * 5
    H = oracle.row_entropy(l)
    np.testing.assert_allclose(H, scipy.stats.entropy(scipy.special.softmax(l, axis=1), axis=1), rtol=1e-12)
    assert oracle.row_entropy(np.zeros((1, 77)))[0] == pytest.approx(np.log(77), rel=1e-14)   # uniform
    one = np.full((1, 50), -np.inf)
    one[0, 3] = 2.0
    assert oracle.row_entropy(one)[0] == 0.0                                                   # one-hot
    # the excluded id: entropy of the vocabulary without it
    keep = [v for v in range(200) if v != 11]
    np.testing.assert_allclose(oracle.row_entropy(l, exclude=11), oracle.row_entropy(l[:, keep]), rtol=1e-13)
    assert (H <= np.log(200) + 1e-12).all() and (H >= 0).all()
