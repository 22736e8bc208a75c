"""Dynamic Contiguous Verification and draft-guided selection (Sections 3.2, 3.3; Algorithm 1).

Readings of the paper used here (the paper is silent or inconsistent on them):
* thresholds are strict: c > tau (Eq. compute_k, Eq. draft_update, Eq. threshold_pd);
* p is the first uncommitted position; positions are absolute, ranges half-open,
  the generation region ends at ``gen_end``;
* the window is clipped at the end: L_eff = min(L, gen_end - p) for K and remasking;
  drafts use the unclipped start p + L;
* K = 0 would stall Algorithm 1, so by default K_eff = max(K, 1) (the top-1 at p
  is committed, i.e. one sequential chain-rule step, Section 2.2); the
  ``no_progress_guard`` flag keeps the literal K;
* a window start whose row carries no statistics (top1 = -1: the row was not scored, which only
  happens when the caller did not re-mask the window) has no prediction to commit: K_eff stays 0
  and the sequence does not advance in that iteration;
* scored rows (``score_all=False``): x_i = [MASK] and p <= i < gen_end (probabilities
  are defined at masked positions, Section 2.1); only those rows can become drafts.
  ``score_all=True``: every position p <= i < gen_end is scored and may be redrafted.
* semi-autoregressive blocks (Section 4 setup: semi-AR remasking with blocks of 32; the paper
  does not say how blocks and the window combine): with ``block_len`` > 0 the generation region is
  cut into blocks of that length starting at ``block_origin``; the decoding window never crosses
  the end of the block that holds p (L_eff = min(L, block_end - p), and the re-mask stops there),
  while drafts keep looking ahead over the whole region from p + L.
"""


def block_end(p: int, gen_end: int, block_origin: int, block_len: int) -> int:
    """End of the semi-AR block holding position p (gen_end without blocks)."""
    if block_len <= 0:
        return gen_end
    return min(gen_end, block_origin + block_len * ((p - block_origin) // block_len + 1))
import numpy as np


def scored_mask(tokens: np.ndarray, p: np.ndarray, gen_end: int, mask_id: int, score_all: bool = False):
    """[B, S] bool: rows whose prediction statistics are computed."""
    B, S = tokens.shape
    idx = np.arange(S)[None, :]
    inside = (idx >= np.asarray(p)[:, None]) & (idx < gen_end)
    return inside if score_all else inside & (tokens == mask_id)


def compute_k(conf_window: np.ndarray, tau_commit: float) -> int:
    """Eq. compute_k: K = sum_{i<L} prod_{j<=i} 1(c_j > tau_commit) over the window's confidences."""
    K = 0
    run = 1
    for c in conf_window:
        run *= 1 if c > tau_commit else 0
        K += run
    return K


def select_contiguous(tokens, p, gen_end, L, tau_commit, tau_draft, mask_id, top1, conf,
                      no_progress_guard=False, score_all=False, contiguous_drafts=False,
                      block_origin=0, block_len=0):
    """One selection step for every sequence: steps (iii)-(iv) of Section 3.3, then (i) for the next.

    tokens [B,S], p [B], top1/conf [B,S] (statistics of the forward on ``tokens``).
    Returns (new tokens, new p, K_raw [B], K_eff [B]); inputs are not modified.
    Per sequence with p < gen_end:
      L_eff = min(L, end - p) with end = gen_end, or the end of p's block with blocks;
      K = Eq. compute_k over conf[p : p + L_eff];
      K_eff = max(K, 1) (unless no_progress_guard, or the row at p has no prediction: top1 = -1);
      commit x[p : p + K_eff] = top1                                 (Algorithm 1, commit)
      for j in [p + L, gen_end): if (x_j = [MASK] or score_all) and conf_j > tau_draft:
          x_j = top1_j                                               (Eq. draft_update)
        with contiguous_drafts (the variant of Appendix E): only the leading chain from p + L
        is drafted: it ends at the first eligible position with conf <= tau_draft; positions
        that already hold a token (not eligible) keep it and do not end the chain
      p += K_eff                                                     (Algorithm 1, advance)
      x[p : min(p + L, end of the new p's block)] = [MASK]           (Eq. remasking, next iteration)
    """
    x = np.array(tokens, dtype=np.int64, copy=True)
    pn = np.array(p, dtype=np.int64, copy=True)
    B, S = x.shape
    K_raw = np.zeros(B, np.int64)
    K_eff = np.zeros(B, np.int64)
    for b in range(B):
        pb = int(pn[b])
        if pb >= gen_end:
            continue
        L_eff = min(L, block_end(pb, gen_end, block_origin, block_len) - pb)
        K = compute_k(conf[b, pb:pb + L_eff], tau_commit)
        has_prediction = top1[b, pb] >= 0
        Ke = K if (no_progress_guard or not has_prediction) else max(K, 1)
        K_raw[b], K_eff[b] = K, Ke
        for j in range(pb, pb + Ke):
            x[b, j] = top1[b, j]
        for j in range(pb + L, gen_end):
            eligible = score_all or tokens[b, j] == mask_id
            if eligible and conf[b, j] > tau_draft:
                x[b, j] = top1[b, j]
            elif eligible and contiguous_drafts:
                break                                     # the chain of Appendix E ends here
        pb += Ke
        pn[b] = pb
        for j in range(pb, min(pb + L, block_end(pb, gen_end, block_origin, block_len))):
            x[b, j] = mask_id
    return x, pn, K_raw, K_eff


def select_noncontiguous(tokens, p, gen_end, L, tau, mask_id, top1, conf, no_progress_guard=False):
    """The non-contiguous threshold rule (Eq. threshold_pd) inside the same sliding window.

    Per sequence with p < gen_end, over the masked positions j of [p, p + L_eff):
      commit x_j = top1_j for every such j with conf_j > tau (independent decisions, Eq. threshold_pd);
      if none qualifies (and not no_progress_guard): commit the one with the highest confidence
      (lowest position on ties) so the loop progresses;
      p <- the first position >= p still holding [MASK] (gen_end if none): the verified prefix.
    No drafts and no remasking: committed tokens past p stay committed.
    Returns (new tokens, new p, K_raw = number passing tau, K_eff = number committed).
    """
    x = np.array(tokens, dtype=np.int64, copy=True)
    pn = np.array(p, dtype=np.int64, copy=True)
    B, S = x.shape
    K_raw = np.zeros(B, np.int64)
    K_eff = np.zeros(B, np.int64)
    for b in range(B):
        pb = int(pn[b])
        if pb >= gen_end:
            continue
        hi = min(pb + L, gen_end)
        cand = [j for j in range(pb, hi) if x[b, j] == mask_id and conf[b, j] >= 0]
        passing = sorted(noncontiguous_commit_set(conf[b], pb, hi, tau) & set(cand))
        commit = list(passing)
        if not commit and cand and not no_progress_guard:
            best = max(cand, key=lambda j: (conf[b, j], -j))
            commit = [best]
        for j in commit:
            x[b, j] = top1[b, j]
        K_raw[b], K_eff[b] = len(passing), len(commit)
        masked = np.nonzero(x[b, pb:gen_end] == mask_id)[0]
        pn[b] = pb + int(masked[0]) if len(masked) else gen_end
    return x, pn, K_raw, K_eff


def noncontiguous_commit_set(conf_row: np.ndarray, lo: int, hi: int, tau: float):
    """Eq. threshold_pd: positions i in [lo, hi) with max-probability c_i > tau."""
    return {i for i in range(lo, hi) if conf_row[i] > tau}
