"""Distribution summary psi, rank head, buckets and branching (oracle).

Test infrastructure: see the package docstring.
"""
from __future__ import annotations

import numpy as np

from .numerics import logsumexp

PSI_DIM = 15
TOPK = 10

# Bucket-to-branching maps recommended in App. A.5 (inference procedure).
BRANCH_MAP_CONCENTRATE = (2, 4, 10, 0)
BRANCH_MAP_FALLBACK = (2, 4, 6, 4)


def bucket_of_rank(r: int) -> int:
    """Rank-head label rule of Sec. 3.3: r = 1 -> b0, 2..4 -> b1,
    5..10 -> b2, > 10 -> b3 (r is 1-based)."""
    if r < 1:
        raise ValueError(r)
    if r == 1:
        return 0
    if r <= 4:
        return 1
    if r <= 10:
        return 2
    return 3


def topk_ids(z, k: int = TOPK) -> np.ndarray:
    """Ids of the k largest logits; larger value first, equal values ordered
    by smaller id (our tie rule; the paper does not state one)."""
    z = np.asarray(z)
    order = np.lexsort((np.arange(z.shape[-1]), -z))
    return order[:k]


def psi(z) -> np.ndarray:
    """15-dim summary of the draft distribution p = softmax(z) (App. B):
    [log p of the top-10 tokens (10), logit gaps top1-rank2, top1-rank3,
    top1-rank5 (3), top-1 probability (1), entropy (1)].

    Natural logarithm, temperature 1, full-vocabulary softmax, gaps in raw
    logits (our reading of the prose description).
    """
    z = np.asarray(z, dtype=np.float64)
    zs = np.sort(z)[::-1]
    lse = logsumexp(z)
    logp = zs[:TOPK] - lse
    gaps = np.array([zs[0] - zs[1], zs[0] - zs[2], zs[0] - zs[4]])
    p = np.exp(z - lse)
    entropy = -np.sum(p * (z - lse))
    return np.concatenate([logp, gaps, [np.exp(logp[0])], [entropy]])


def rank_scores(rank_w, rank_b, h_last, psi_vec) -> np.ndarray:
    """Rank head g_phi of Eq. 4 read as one linear layer with bias over
    [h^(L), psi] (the paper fixes its inputs and four outputs only)."""
    x = np.concatenate([np.asarray(h_last, np.float64), psi_vec])
    return np.asarray(rank_w, np.float64) @ x + np.asarray(rank_b, np.float64)


def bucket_of_scores(scores) -> int:
    """argmax over the four buckets, ties to the lower bucket."""
    return int(np.argmax(scores))
