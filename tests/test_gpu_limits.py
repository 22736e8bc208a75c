"""Size limits of dcl_denoise_step (include/dcl.h): B*S <= 2^22 tokens; q/k/v^T of one step below
2^31 elements and every GEMM activation operand below 2^31 elements (the kernels' 32-bit offsets).

* The largest accepted batch of 4096-token sequences of the small model (681 sequences, 2.79 M
  tokens, where its q/k/v^T reach 2^31 - 2.4 M elements) runs: its scored-row set is exactly the
  masked positions past p in every sequence, every scored row's statistics are well-formed, two
  sampled sequences (first and last, whose offsets are the largest) match the oracle within the
  whole-step tolerance, and the selection is bit-exact on the GPU's own statistics for every
  sequence.
The rejections past these limits (one sequence more, B*S above 2^22, a geometry whose FFN activations
would pass 2^31 elements) are host-only checks made before anything touches the device; they are
tested without a GPU in test_abi.py."""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from oracle.numerics import WeightView

from helpers import compare_stats, derived_tolerance, runner_for, stats_to_np, to_dev

pytestmark = pytest.mark.gpu

_C1 = synth.WORKLOADS["c1"]
# 681 sequences of 4096 tokens: 64 prompt tokens, draft stand-ins at [96, 160), the rest masked.
# 681 * (4096 + 8) * 768 q/k/v^T rows = 2^31 - 2.4 M; 682 sequences pass 2^31.
_MAX = dataclasses.replace(_C1, key="max_tokens", batch=681, prompt_len=64, gen_len=4032, window=32, p=64,
                           draft=(96, 160))


def test_largest_step_matches_oracle_on_sampled_sequences():
    import torch
    import paper_2607_20467_amd as dcl
    w = _MAX
    g = w.geom
    qkv_rows = (g.n_heads + 2 * g.n_kv_heads) * g.head_dim
    assert w.batch * (w.seq + 8) * qkv_rows < 1 << 31 <= (w.batch + 1) * (w.seq + 8) * qkv_rows
    stored = synth.make_weights(g)
    W = WeightView(stored)
    run = runner_for(w, stored)
    tok, p = synth.initial_state(w)
    B, S = tok.shape
    print(f"case max_tokens: B={B} S={S} workspace {run.workspace(B, S)[1] / 2**30:.1f} GiB", flush=True)
    t_dev, p_dev = to_dev(tok), to_dev(p)
    st = stats_to_np(run.step(t_dev, p_dev, w.gen_end))
    print("step done", flush=True)

    pos = np.arange(S)[None]
    scored = (tok == g.mask_id) & (pos >= p[:, None]) & (pos < w.gen_end)
    np.testing.assert_array_equal(st["conf"] >= 0, scored)
    np.testing.assert_array_equal(st["top1"][~scored], -1)
    np.testing.assert_array_equal(st["conf"][~scored], -1.0)
    c, p2, lse = st["conf"][scored], st["p2"][scored], st["lse"][scored]
    t1, t2 = st["top1"][scored], st["top2"][scored]
    assert np.isfinite(lse).all() and (c > 0).all() and (c <= 1).all() and (p2 >= 0).all() and (p2 <= c).all()
    assert ((t1 >= 0) & (t1 < g.vocab) & (t2 >= 0) & (t2 < g.vocab) & (t1 != t2)).all()
    # the vocabulary holds 4096 ids, so the top-1 probability is at least 1/4096
    assert (c >= 1.0 / g.vocab * (1 - 1e-6)).all()

    for b in (0, B - 1):
        print(f"oracle on sequence {b}", flush=True)
        ref = oracle.step(g, W, tok[b:b + 1], p[b:b + 1], w.gen_end)
        ct, lt = derived_tolerance(g, W, tok[b:b + 1], p[b:b + 1], w.gen_end, ref)
        rep = compare_stats({k: v[b:b + 1] for k, v in st.items()}, ref, w.tau_commit, w.tau_draft,
                            what=f"max_tokens[{b}]", conf_tol=ct, logit_tol=lt)
        print(f"max_tokens[{b}]", rep, flush=True)

    kr = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    ke = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    stats_dev = {k: torch.from_numpy(v).cuda() for k, v in st.items()}
    dcl.dcl_select_contiguous(t_dev, B, S, p_dev, w.gen_end, w.window, w.tau_commit, w.tau_draft, g.mask_id,
                              stats_dev, kr, ke)
    torch.cuda.synchronize()
    x_ref, p_ref, kr_ref, ke_ref = oracle.select_contiguous(tok, p, w.gen_end, w.window, w.tau_commit, w.tau_draft,
                                                            g.mask_id, st["top1"], st["conf"].astype(np.float64))
    np.testing.assert_array_equal(t_dev.cpu().numpy(), x_ref)
    np.testing.assert_array_equal(p_dev.cpu().numpy(), p_ref)
    np.testing.assert_array_equal(kr.cpu().numpy(), kr_ref)
    np.testing.assert_array_equal(ke.cpu().numpy(), ke_ref)
    del run, stats_dev
    torch.cuda.empty_cache()
