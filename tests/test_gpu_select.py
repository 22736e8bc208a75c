"""GPU parity of dcl_select_contiguous (DCV, commit, drafts, remask) against the oracle: bit-exact."""
import numpy as np
import pytest

import oracle
from oracle.select import scored_mask

pytestmark = pytest.mark.gpu


def _run_gpu(tok, p, end, L, tc, td, mask, top1, conf, flags=0, p2=None, block_origin=0, block_len=0):
    import torch
    import paper_2607_20467_amd as dcl
    B, S = tok.shape
    t = torch.from_numpy(tok.astype(np.int32)).cuda()
    pp = torch.from_numpy(p.astype(np.int32)).cuda()
    st = {"top1": torch.from_numpy(top1.astype(np.int32)).cuda(),
          "top2": torch.zeros((B, S), dtype=torch.int32, device="cuda"),
          "conf": torch.from_numpy(conf.astype(np.float32)).cuda(),
          "p2": (torch.zeros((B, S), dtype=torch.float32) if p2 is None else torch.from_numpy(p2.astype(np.float32))).cuda(),
          "lse": torch.zeros((B, S), dtype=torch.float32, device="cuda")}
    kr = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    ke = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    dcl.dcl_select_contiguous(t, B, S, pp, end, L, tc, td, mask, st, kr, ke, flags, block_origin=block_origin,
                              block_len=block_len)
    torch.cuda.synchronize()
    return t.cpu().numpy(), pp.cpu().numpy(), kr.cpu().numpy(), ke.cpu().numpy()


@pytest.mark.parametrize("seed", range(6))
def test_select_random_states_bit_exact(seed):
    rng = np.random.default_rng(100 + seed)
    mask = 4095
    B, S = int(rng.integers(1, 9)), int(rng.integers(8, 700))
    end = int(rng.integers(1, S + 1))
    L = int(rng.choice([1, 2, 16, 32, 64, 128, 300]))
    tok = rng.integers(0, 4000, (B, S))
    p = rng.integers(0, end + 1, B)
    p[0] = min(p[0], end - 1)
    for b in range(B):
        tok[b, p[b]:] = np.where(rng.random(S - p[b]) < 0.6, mask, tok[b, p[b]:])
        tok[b, p[b]:min(p[b] + L, end)] = mask                     # the window is masked before a step
    for flags, score_all in ((0, False), (1, False), (2, True), (3, True)):
        sc = scored_mask(tok, p, end, mask, score_all)
        # float32 confidences, compared identically by both sides
        conf = np.where(sc, rng.uniform(0, 1, (B, S)).astype(np.float32), np.float32(-1)).astype(np.float32)
        conf[sc & (rng.random((B, S)) < 0.05)] = np.float32(0.7)   # exact ties with the threshold
        top1 = np.where(sc, rng.integers(0, 4000, (B, S)), -1)
        tc, td = np.float32(0.7), np.float32(rng.choice([0.5, 0.9, 0.98, 1.5]))
        ref = oracle.select_contiguous(tok, p, end, L, float(tc), float(td), mask, top1, conf.astype(np.float64),
                                       no_progress_guard=bool(flags & 1), score_all=score_all)
        got = _run_gpu(tok, p, end, L, float(tc), float(td), mask, top1, conf, flags)
        for name, g, r in zip(("tokens", "p", "K_raw", "K_eff"), got, ref):
            np.testing.assert_array_equal(g, r, err_msg=f"{name} flags={flags} B={B} S={S} L={L} end={end}")


def test_select_golden_cases():
    import json
    import os
    cases = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "select_cases.json")))["select_cases"]
    for c in cases:
        got = _run_gpu(np.array([c["tokens"]]), np.array([c["p"]]), c["gen_end"], c["L"], c["tau_commit"],
                       c["tau_draft"], c["mask_id"], np.array([c["top1"]]), np.array([c["conf"]], np.float32),
                       block_origin=c.get("block_origin", 0), block_len=c.get("block_len", 0))
        assert got[0][0].tolist() == c["expect_tokens"], c["name"]
        assert (got[1][0], got[2][0], got[3][0]) == (c["expect_p"], c["expect_K_raw"], c["expect_K_eff"]), c["name"]


@pytest.mark.parametrize("seed", range(6))
def test_selection_variants_bit_exact(seed):
    """DCL_SEL_NONCONTIGUOUS (Eq. threshold_pd in the window) and DCL_SEL_CONTIGUOUS_DRAFTS (Appendix E)
    against the oracle's rules on random states, with exact threshold ties and confidence ties."""
    import paper_2607_20467_amd as dcl
    rng = np.random.default_rng(500 + seed)
    mask = 4095
    B, S = int(rng.integers(1, 9)), int(rng.integers(8, 700))
    end = int(rng.integers(1, S + 1))
    L = int(rng.choice([1, 2, 16, 32, 64, 128, 300]))
    tok = rng.integers(0, 4000, (B, S))
    p = rng.integers(0, end + 1, B)
    p[0] = min(p[0], end - 1)
    for b in range(B):
        tok[b, p[b]:] = np.where(rng.random(S - p[b]) < 0.6, mask, tok[b, p[b]:])
    NC, CD, NG, SA = dcl.DCL_SEL_NONCONTIGUOUS, dcl.DCL_SEL_CONTIGUOUS_DRAFTS, 1, 2
    for flags in (NC, NC | NG, CD, CD | NG, CD | SA):
        score_all = bool(flags & SA)
        t = tok.copy()
        if not flags & NC:
            for b in range(B):
                t[b, p[b]:min(p[b] + L, end)] = mask
        sc = scored_mask(t, p, end, mask, score_all)
        conf = np.where(sc, rng.uniform(0, 1, (B, S)).astype(np.float32), np.float32(-1)).astype(np.float32)
        conf[sc & (rng.random((B, S)) < 0.05)] = np.float32(0.7)   # ties with tau_commit
        conf[sc & (rng.random((B, S)) < 0.05)] = np.float32(0.25)  # ties between rows (non-contiguous guard)
        if flags & CD:                                            # long passing runs so chains matter
            for b in range(B):
                lo = int(rng.integers(0, S))
                hi = min(S, lo + int(rng.integers(1, 80)))
                conf[b, lo:hi] = np.where(sc[b, lo:hi], np.float32(0.99), np.float32(-1))
        top1 = np.where(sc, rng.integers(0, 4000, (B, S)), -1)
        tc, td = np.float32(0.7), np.float32(rng.choice([0.3, 0.5, 0.9]))
        if flags & NC:
            ref = oracle.select_noncontiguous(t, p, end, L, float(tc), mask, top1, conf.astype(np.float64),
                                              no_progress_guard=bool(flags & NG))
        else:
            ref = oracle.select_contiguous(t, p, end, L, float(tc), float(td), mask, top1, conf.astype(np.float64),
                                           no_progress_guard=bool(flags & NG), score_all=score_all,
                                           contiguous_drafts=True)
        got = _run_gpu(t, p, end, L, float(tc), float(td), mask, top1, conf, flags)
        for name, g, r in zip(("tokens", "p", "K_raw", "K_eff"), got, ref):
            np.testing.assert_array_equal(g, r, err_msg=f"{name} flags={flags} B={B} S={S} L={L} end={end}")



@pytest.mark.parametrize("seed", range(4))
def test_margin_acceptance_bit_exact(seed):
    """DCL_SEL_MARGIN: every rule applied to the float32 margin conf - p2 (unscored rows -1) equals the
    oracle's rule applied to the same float32 values."""
    import paper_2607_20467_amd as dcl
    rng = np.random.default_rng(900 + seed)
    mask = 4095
    B, S = int(rng.integers(1, 6)), int(rng.integers(8, 500))
    end = int(rng.integers(1, S + 1))
    L = int(rng.choice([1, 16, 32, 100]))
    tok = rng.integers(0, 4000, (B, S))
    p = rng.integers(0, end + 1, B)
    p[0] = min(p[0], end - 1)
    for b in range(B):
        tok[b, p[b]:] = np.where(rng.random(S - p[b]) < 0.6, mask, tok[b, p[b]:])
    MG = dcl.DCL_SEL_MARGIN
    for flags in (MG, MG | dcl.DCL_SEL_CONTIGUOUS_DRAFTS, MG | dcl.DCL_SEL_NONCONTIGUOUS):
        t = tok.copy()
        if not flags & dcl.DCL_SEL_NONCONTIGUOUS:
            for b in range(B):
                t[b, p[b]:min(p[b] + L, end)] = mask
        sc = scored_mask(t, p, end, mask)
        c = rng.uniform(0.3, 1.0, (B, S)).astype(np.float32)
        q = (c * rng.uniform(0, 1, (B, S))).astype(np.float32)          # p2 <= conf
        q[rng.random((B, S)) < 0.05] = np.float32(0.1)
        c[rng.random((B, S)) < 0.05] = np.float32(0.6)                 # margin ties with tau: 0.6 - 0.1 = 0.5
        conf = np.where(sc, c, np.float32(-1)).astype(np.float32)
        p2 = np.where(sc, q, np.float32(-1)).astype(np.float32)
        marg = np.where(sc, (conf - p2).astype(np.float32), np.float32(-1)).astype(np.float64)
        top1 = np.where(sc, rng.integers(0, 4000, (B, S)), -1)
        tc, td = 0.5, float(np.float32(rng.choice([0.3, 0.5, 0.8])))
        if flags & dcl.DCL_SEL_NONCONTIGUOUS:
            ref = oracle.select_noncontiguous(t, p, end, L, tc, mask, top1, marg)
        else:
            ref = oracle.select_contiguous(t, p, end, L, tc, td, mask, top1, marg,
                                           contiguous_drafts=bool(flags & dcl.DCL_SEL_CONTIGUOUS_DRAFTS))
        got = _run_gpu(t, p, end, L, tc, td, mask, top1, conf, flags, p2=p2)
        for name, g, r in zip(("tokens", "p", "K_raw", "K_eff"), got, ref):
            np.testing.assert_array_equal(g, r, err_msg=f"{name} flags={flags} B={B} S={S} L={L} end={end}")


@pytest.mark.parametrize("tc,L", [(0.0, 1), (0.0, 5000), (1.0, 1), (1.0, 5000), (0.7, 5000)])
def test_select_degenerate_thresholds_and_windows(tc, L):
    """tau_c = 0: every scored window row passes, K = L_eff; tau_c = 1: none passes, K = 0 and the
    progress guard commits one token (K_eff = 1); a window longer than the remaining region is
    clipped to gen_end - p; L = 1 is the sequential decoder. Bit-exact against the oracle."""
    rng = np.random.default_rng(int(tc * 10) + L)
    mask = 4095
    B, S = 5, 333
    end = 300
    tok = rng.integers(0, 4000, (B, S))
    p = np.array([0, 17, 150, 299, 300])
    for b in range(B):
        tok[b, p[b]:] = np.where(rng.random(S - p[b]) < 0.7, mask, tok[b, p[b]:])
        tok[b, p[b]:min(p[b] + L, end)] = mask
    sc = scored_mask(tok, p, end, mask, False)
    conf = np.where(sc, rng.uniform(1e-4, 1, (B, S)).astype(np.float32), np.float32(-1)).astype(np.float32)
    top1 = np.where(sc, rng.integers(0, 4000, (B, S)), -1)
    ref = oracle.select_contiguous(tok, p, end, L, tc, 0.98, mask, top1, conf.astype(np.float64))
    got = _run_gpu(tok, p, end, L, tc, 0.98, mask, top1, conf)
    for name, g, r in zip(("tokens", "p", "K_raw", "K_eff"), got, ref):
        np.testing.assert_array_equal(g, r, err_msg=f"{name} tc={tc} L={L}")
    live = p < end
    l_eff = np.minimum(L, end - p)
    if tc == 0.0:
        np.testing.assert_array_equal(got[2][live], l_eff[live])
    if tc == 1.0:
        np.testing.assert_array_equal(got[2][live], 0)
        np.testing.assert_array_equal(got[3][live], 1)
    np.testing.assert_array_equal(got[1][~live], p[~live])      # a finished sequence does not move


@pytest.mark.parametrize("seed", range(4))
def test_select_with_semi_ar_blocks_bit_exact(seed):
    """Semi-autoregressive blocks (reading R24): the window and its re-mask stop at the end of p's block,
    with blocks shorter and longer than the window, origins before and inside the state, every flag."""
    rng = np.random.default_rng(300 + seed)
    mask = 4095
    B, S = int(rng.integers(1, 9)), int(rng.integers(16, 600))
    end = int(rng.integers(8, S + 1))
    L = int(rng.choice([1, 8, 16, 32, 128]))
    BL = int(rng.choice([1, 5, 16, 32, 64]))
    origin = int(rng.integers(0, end))
    tok = rng.integers(0, 4000, (B, S))
    p = rng.integers(max(origin - 3, 0), end + 1, B)
    for b in range(B):
        tok[b, p[b]:] = np.where(rng.random(S - p[b]) < 0.6, mask, tok[b, p[b]:])
        tok[b, p[b]:min(p[b] + L, end)] = mask
    for flags, score_all in ((0, False), (1, False), (2, True)):
        sc = scored_mask(tok, p, end, mask, score_all)
        conf = np.where(sc, rng.uniform(0, 1, (B, S)).astype(np.float32), np.float32(-1)).astype(np.float32)
        conf[sc & (rng.random((B, S)) < 0.05)] = np.float32(0.7)
        top1 = np.where(sc, rng.integers(0, 4000, (B, S)), -1)
        tc, td = np.float32(0.7), np.float32(rng.choice([0.5, 0.9, 1.5]))
        ref = oracle.select_contiguous(tok, p, end, L, float(tc), float(td), mask, top1, conf.astype(np.float64),
                                       no_progress_guard=bool(flags & 1), score_all=score_all,
                                       block_origin=origin, block_len=BL)
        got = _run_gpu(tok, p, end, L, float(tc), float(td), mask, top1, conf, flags, block_origin=origin,
                       block_len=BL)
        for name, g, r in zip(("tokens", "p", "K_raw", "K_eff"), got, ref):
            np.testing.assert_array_equal(g, r, err_msg=f"{name} flags={flags} B={B} S={S} L={L} blocks {origin}+{BL}")
