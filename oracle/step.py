"""One denoising iteration's forward + statistics (Algorithm 1, Forward; Section 2.1).

``step`` returns, for every sequence and position, the prediction statistics of
the scored rows (``select.scored_mask``) and sentinels elsewhere:
top1/top2 = -1, conf/p2 = -1, lse = 0.
"""
import numpy as np

from .forward import forward, lm_logits
from .scores import SENTINEL_CONF, SENTINEL_ID, row_entropy, row_stats
from .select import scored_mask


def step(geom, weights, tokens, p, gen_end, kv=None, score_all=False, bf16_boundary=True,
         rope=True, return_logits_rows=None, dtype=np.float64, return_hidden=False, suppress_mask=False):
    """Statistics dict with arrays [B, S]: top1, top2, conf, p2, lse.

    kv: optional callable (b, layer) -> (Kc [Hkv,P,dh], Vc [Hkv,dh,P]) with prefix length ``kv_prefix``
        given as attribute ``kv.prefix``; tokens are then at absolute positions prefix + i.
    return_logits_rows: optional list of flat row indices b*S+i whose float64 logits are also returned
        (key "logits", [len, V]); they need not be scored rows.
    dtype: arithmetic of the evaluation (float64 = the oracle; float32 only sizes tolerances).
    return_hidden: also return the final hidden states h_f [B, S, d] (key "hidden").
    suppress_mask: the [MASK] id is removed from the vocabulary of the statistics (``row_stats``).
    """
    tokens = np.asarray(tokens)
    B, S = tokens.shape
    sc = scored_mask(tokens, p, gen_end, geom.mask_id, score_all)
    out = {
        "top1": np.full((B, S), SENTINEL_ID, np.int64),
        "top2": np.full((B, S), SENTINEL_ID, np.int64),
        "conf": np.full((B, S), SENTINEL_CONF),
        "p2": np.full((B, S), SENTINEL_CONF),
        "lse": np.zeros((B, S)),
        "entropy": np.full((B, S), SENTINEL_CONF),
    }
    want = {} if return_logits_rows is None else {int(r): n for n, r in enumerate(return_logits_rows)}
    logits_out = None if return_logits_rows is None else np.empty((len(want), geom.vocab))
    hidden = np.zeros((B, S, geom.d_model)) if return_hidden else None
    prefix = 0 if kv is None else kv.prefix
    pos = prefix + np.arange(S)
    for b in range(B):
        extra = [i for i in range(S) if (b * S + i) in want]
        rows = np.nonzero(sc[b])[0]
        if len(rows) == 0 and not extra and not return_hidden:
            continue
        kvb = None if kv is None else (lambda l, b=b: kv(b, l))
        hf = forward(geom, weights, tokens[b], pos, kv=kvb, bf16_boundary=bf16_boundary, rope=rope, dtype=dtype)
        if return_hidden:
            hidden[b] = hf
        if len(rows):
            lg = lm_logits(weights, hf[rows], dtype=dtype)
            ex = geom.mask_id if suppress_mask else None
            t1, t2, c, p2, lse = row_stats(lg, exclude=ex)
            out["entropy"][b, rows] = row_entropy(lg, exclude=ex)
            out["top1"][b, rows] = t1
            out["top2"][b, rows] = t2
            out["conf"][b, rows] = c
            out["p2"][b, rows] = p2
            out["lse"][b, rows] = lse
        if extra:
            lg = lm_logits(weights, hf[extra], dtype=dtype)
            for n, i in enumerate(extra):
                logits_out[want[b * S + i]] = lg[n]
    if logits_out is not None:
        out["logits"] = logits_out
    if return_hidden:
        out["hidden"] = hidden
    return out


def step_from_weights(workload, weights, tokens, p, kv=None, score_all=False, **kw):
    """``step`` with geometry and generation end taken from a ``synth.Workload``."""
    return step(workload.geom, weights, tokens, p, workload.gen_end, kv=kv, score_all=score_all, **kw)
