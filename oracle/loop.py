"""Full decode loops (Algorithm 1, Appendix A) and the reference decoders used as pins.

``generate``           Algorithm 1: remask window, forward, K (Eq. compute_k), commit, drafts, advance.
``sequential_greedy``  chain-rule decoding (Section 2.2, Eq. sequential_chain): one forward per token,
                       commit the top-1 at the leftmost masked position.
``noncontiguous_commit_set``  positions a threshold rule commits independently (Eq. threshold_pd).
"""
import numpy as np

from .select import block_end, noncontiguous_commit_set, select_contiguous  # noqa: F401
from .step import step


def generate(geom, weights, prompt, gen_len, L, tau_commit, tau_draft, no_progress_guard=False,
             score_all=False, max_steps=None, trace=None, block_len=0):
    """Algorithm 1 for one batch of prompts [B, N]; returns (tokens [B, N+M], steps).

    x = prompt || [MASK]^M, p = N; while any p < N+M: one ``step`` then ``select_contiguous``
    (whose final remask is the loop-top draft invalidation of the next iteration).
    ``trace`` (a list) receives (tokens, p, K_raw, K_eff) after every iteration.
    ``block_len`` > 0: semi-autoregressive blocks of that length from N (``select.block_end``): the
    window and its re-mask stay inside the block holding p.
    """
    prompt = np.asarray(prompt)
    B, N = prompt.shape
    end = N + gen_len
    x = np.full((B, end), geom.mask_id, np.int64)
    x[:, :N] = prompt
    p = np.full(B, N, np.int64)
    steps = 0
    limit = gen_len if max_steps is None else max_steps
    while (p < end).any():
        if steps >= limit:
            raise RuntimeError("decode loop exceeded %d steps" % limit)
        for b in range(B):                      # draft invalidation before the forward
            x[b, p[b]:min(p[b] + L, block_end(p[b], end, N, block_len))] = geom.mask_id
        st = step(geom, weights, x, p, end, score_all=score_all)
        x, p, k_raw, k_eff = select_contiguous(x, p, end, L, tau_commit, tau_draft, geom.mask_id,
                                               st["top1"], st["conf"], no_progress_guard, score_all,
                                               block_origin=N, block_len=block_len)
        steps += 1
        if trace is not None:
            trace.append((x.copy(), p.copy(), k_raw, k_eff))
    return x, steps


def sequential_greedy(geom, weights, prompt, gen_len):
    """Chain-rule greedy decoding: M forwards; each commits the top-1 at the first masked position."""
    prompt = np.asarray(prompt)
    B, N = prompt.shape
    end = N + gen_len
    x = np.full((B, end), geom.mask_id, np.int64)
    x[:, :N] = prompt
    for t in range(gen_len):
        i = N + t
        p = np.full(B, i, np.int64)
        st = step(geom, weights, x, p, end)
        x[:, i] = st["top1"][:, i]
    return x

