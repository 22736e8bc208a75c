"""Per-position prediction statistics (Section 2.1, Eq. 2 and Eq. threshold_pd; Section 2.2).

For a logit row l over the vocabulary V:
  P(x_i = v) = softmax(l)_v                                   (Eq. 2)
  x_hat_i = argmax_v P, c_i = max_v P                          (top-1 token, confidence)
  second-ranked token and its probability                      (the top-1/top-2 gap of Section 2.2)
Ties go to the lowest token id (greedy decoding, Section 4 setup; the paper
does not specify a tie rule). The [MASK] id is an ordinary member of V unless
``exclude`` names it: an excluded id takes no probability mass and is never
ranked (its logit counts as -inf), i.e. the statistics of the softmax over V
without that id.
"""
import numpy as np

SENTINEL_ID = -1      # top1/top2 of rows that are not scored
SENTINEL_CONF = -1.0  # conf/p2 of rows that are not scored


def row_stats(logits: np.ndarray, exclude=None):
    """Statistics of each row of ``logits`` [R, V] (float64).

    Returns (top1 [R] int64, top2 [R] int64, conf [R], p2 [R], lse [R]) where
    conf = P(top1), p2 = P(top2) and lse = log sum_v exp(l_v).
    Computed from the materialised softmax and a stable sort on (-l, id).
    exclude: optional token id removed from the vocabulary (logit -inf).
    """
    l = np.array(logits, dtype=np.float64, copy=True)
    if exclude is not None:
        l[:, int(exclude)] = -np.inf
    R, V = l.shape
    order = np.argsort(-l, axis=1, kind="stable")      # equal values keep ascending id order
    top1 = order[:, 0]
    top2 = order[:, 1]
    m = l[np.arange(R), top1]
    e = np.exp(l - m[:, None])
    z = e.sum(axis=1)
    P = e / z[:, None]
    conf = P[np.arange(R), top1]
    p2 = P[np.arange(R), top2]
    lse = m + np.log(z)
    return top1, top2, conf, p2, lse


def row_entropy(logits: np.ndarray, exclude=None):
    """Entropy of each row's softmax, H = -sum_v P log P (Section 2.2: the marginal entropies H(x_i | C)
    of the parallel-decoding error bound), over V without ``exclude`` if given. Natural log.
    """
    l = np.array(logits, dtype=np.float64, copy=True)
    if exclude is not None:
        l[:, int(exclude)] = -np.inf
    m = l.max(axis=1, keepdims=True)
    e = np.exp(l - m)
    z = e.sum(axis=1, keepdims=True)
    P = e / z
    logP = np.where(P > 0, (l - m) - np.log(z), 0.0)
    return -(P * logP).sum(axis=1)
