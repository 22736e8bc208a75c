"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI, run the oracle,
compare with the tolerances of the build's parity bar."""
import numpy as np

import synth

CONF_TOL = 1e-3        # max-abs on confidences
LOGIT_TOL = 2e-2       # max-abs on float32 logits vs the float64 oracle
NEAR = 1e-3            # |conf - tau| below this is reported separately (not a mismatch)
TIE_GAP = 4e-2         # logit gap top1 - top2 below this: token id may legitimately flip


def runner_for(workload, stored, max_positions=None, rope=True):
    """Runner over the synth weights (numpy, load order of include/dcl.h)."""
    from paper_2607_20467_amd import Runner
    names = [n for n, _, _ in synth.tensor_specs(workload.geom)]
    tensors = [stored[n] for n in names]
    mp = max_positions or max(4096, workload.kv_prefix + workload.seq)
    return Runner(workload.geom, tensors, max_positions=mp, rope_enabled=rope)


def to_dev(a, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def stats_to_np(st):
    import torch
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in st.items()}


def compare_stats(gpu, ref, tau_c=None, tau_d=None, what=""):
    """Parity of one step's statistics. Returns a report dict; asserts the bar."""
    scored = ref["conf"] >= 0
    np.testing.assert_array_equal(gpu["conf"] >= 0, scored, err_msg=f"{what}: scored-row sets differ")
    np.testing.assert_array_equal(gpu["top1"][~scored], -1)
    np.testing.assert_array_equal(gpu["conf"][~scored], -1.0)
    dc = np.abs(gpu["conf"][scored] - ref["conf"][scored])
    gap = np.log(np.maximum(ref["conf"][scored], 1e-300)) - np.log(np.maximum(ref["p2"][scored], 1e-300))
    tie = gap < TIE_GAP
    id_bad = (gpu["top1"][scored] != ref["top1"][scored]) & ~tie
    near = np.zeros_like(tie)
    for tau in (tau_c, tau_d):
        if tau is not None:
            near |= np.abs(ref["conf"][scored] - tau) < NEAR
    rep = {"rows": int(scored.sum()), "conf_max_abs": float(dc.max()) if dc.size else 0.0,
           "near_tie": int(tie.sum()), "near_threshold": int(near.sum()),
           "top1_mismatch": int((gpu["top1"][scored] != ref["top1"][scored]).sum())}
    print(what, rep, flush=True)
    assert dc.size == 0 or dc.max() <= CONF_TOL, f"{what}: conf max-abs {dc.max():.3g} > {CONF_TOL}"
    assert not id_bad.any(), f"{what}: top1 mismatch at {np.nonzero(id_bad)[0][:10]} (not near-tie)"
    dl = np.abs(gpu["lse"][scored] - ref["lse"][scored])
    assert dl.size == 0 or dl.max() <= LOGIT_TOL, f"{what}: lse max-abs {dl.max():.3g}"
    return rep
