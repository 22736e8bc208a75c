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
* scored rows (``score_all=False``): x_i = [MASK] and p <= i < gen_end (probabilities
  are defined at masked positions, Section 2.1); only those rows can become drafts.
  ``score_all=True``: every position p <= i < gen_end is scored and may be redrafted.
"""
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
                      no_progress_guard=False, score_all=False):
    """One selection step for every sequence: steps (iii)-(iv) of Section 3.3, then (i) for the next.

    tokens [B,S], p [B], top1/conf [B,S] (statistics of the forward on ``tokens``).
    Returns (new tokens, new p, K_raw [B], K_eff [B]); inputs are not modified.
    Per sequence with p < gen_end:
      L_eff = min(L, gen_end - p); K = Eq. compute_k over conf[p : p + L_eff];
      K_eff = max(K, 1) (unless no_progress_guard);
      commit x[p : p + K_eff] = top1                                 (Algorithm 1, commit)
      for j in [p + L, gen_end): if (x_j = [MASK] or score_all) and conf_j > tau_draft:
          x_j = top1_j                                               (Eq. draft_update)
      p += K_eff                                                     (Algorithm 1, advance)
      x[p : min(p + L, gen_end)] = [MASK]                            (Eq. remasking, next iteration)
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
        L_eff = min(L, gen_end - pb)
        K = compute_k(conf[b, pb:pb + L_eff], tau_commit)
        Ke = K if no_progress_guard else max(K, 1)
        K_raw[b], K_eff[b] = K, Ke
        for j in range(pb, pb + Ke):
            x[b, j] = top1[b, j]
        for j in range(pb + L, gen_end):
            eligible = score_all or tokens[b, j] == mask_id
            if eligible and conf[b, j] > tau_draft:
                x[b, j] = top1[b, j]
        pb += Ke
        pn[b] = pb
        for j in range(pb, min(pb + L, gen_end)):
            x[b, j] = mask_id
    return x, pn, K_raw, K_eff
