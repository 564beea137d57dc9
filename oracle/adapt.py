"""Head-only serving-time update of the drafter (oracle).

Test infrastructure: see the package docstring.

Sec. 3.4 and the per-query adaptation algorithm of App. A.3: the verifier
marks rejected positions; they are buffered, and when the head buffer
saturates the "head-only" action steps the drafter's LM head and rank head
(the decoder trunk stays frozen) on the adaptation loss plus
lambda KL(p_train || p_0) against the pre-deployment drafter, on a training
copy of the weights, on a separate stream.  The bandit that chooses the
action is not part of this.

Readings (the paper names the pieces, not their formulas):
* a buffered position is (h^(L) of the drafter row that predicted it, the
  token the target chose there); the LM-head operand is the drafter's own
  a = norm_final(h^(L)) (bf16-rounded in the bf16 configurations);
* adaptation loss = cross-entropy of the drafter distribution
  p = softmax(W_lm a) against the target's token (skipped for a token
  outside a reduced drafter vocabulary) + cross-entropy of the rank head
  softmax(W_r [h^(L), psi] + b_r) against the bucket of that token's rank
  in p (Sec. 3.3 rule; a token outside the vocabulary ranks past 10);
  psi and the rank label are taken from p before the step and held fixed;
* the KL term compares the full distributions p and p_0 = softmax(W_lm0 a);
* the mean over positions, one plain SGD step of rate lr; the updated LM
  head is rounded back to its storage precision.
"""
from __future__ import annotations

import numpy as np

from .numerics import Numerics, logsumexp, rmsnorm
from .rank import bucket_of_rank, psi as psi_of


def lm_operand(h, final_norm, eps, num: Numerics):
    return num.act(rmsnorm(np.asarray(h, np.float64), final_norm, eps))


def target_rank(z, idx):
    """1-based rank of drafter id idx in logits z (larger first, equal
    logits ordered by smaller id); None (past every rank) when idx is None."""
    if idx is None:
        return None
    z = np.asarray(z)
    return int(np.sum(z > z[idx]) + np.sum((z == z[idx])[:idx]) + 1)


def drafter_id(d2t, token):
    if d2t is None:
        return int(token)
    i = int(np.searchsorted(d2t, token))
    return i if i < len(d2t) and d2t[i] == token else None


def prepare(lm_w, h, targets, final_norm, eps, num, d2t=None):
    """Operands, fixed psi and fixed rank labels of a buffered batch."""
    A = lm_operand(h, final_norm, eps, num)
    Z = A @ np.asarray(lm_w, np.float64).T
    ids = [drafter_id(d2t, y) for y in targets]
    psis = np.stack([psi_of(z) for z in Z])
    buckets = []
    for z, i in zip(Z, ids):
        r = target_rank(z, i)
        buckets.append(3 if r is None else bucket_of_rank(r))
    return A, ids, psis, np.array(buckets)


def head_loss(lm_w, rank_w, rank_b, lm_w0, A, h, ids, psis, buckets,
              kl_weight):
    """Mean adaptation loss + lambda KL of a batch, with psi and the rank
    labels held fixed."""
    lm_w = np.asarray(lm_w, np.float64)
    Z = A @ lm_w.T
    Z0 = A @ np.asarray(lm_w0, np.float64).T
    X = np.concatenate([np.asarray(h, np.float64), psis], axis=1)
    S = X @ np.asarray(rank_w, np.float64).T + np.asarray(rank_b, np.float64)
    total = 0.0
    for i in range(len(A)):
        lse, lse0 = logsumexp(Z[i]), logsumexp(Z0[i])
        logp, logp0 = Z[i] - lse, Z0[i] - lse0
        if ids[i] is not None:
            total -= logp[ids[i]]
        total += kl_weight * float(np.sum(np.exp(logp) * (logp - logp0)))
        total -= S[i][buckets[i]] - logsumexp(S[i])
    return total / len(A)


def logit_grads(lm_w, lm_w0, A, ids, kl_weight):
    """Gradient of head_loss with respect to the LM logits z_i = W_lm a_i
    (rows already divided by the batch size)."""
    Z = A @ np.asarray(lm_w, np.float64).T
    Z0 = A @ np.asarray(lm_w0, np.float64).T
    n = len(A)
    G = np.zeros_like(Z)
    for i in range(n):
        logp = Z[i] - logsumexp(Z[i])
        logp0 = Z0[i] - logsumexp(Z0[i])
        p = np.exp(logp)
        g = np.zeros_like(p)
        if ids[i] is not None:
            g += p
            g[ids[i]] -= 1.0
        kl = float(np.sum(p * (logp - logp0)))
        g += kl_weight * p * (logp - logp0 - kl)
        G[i] = g / n
    return G


def head_grads(lm_w, rank_w, rank_b, lm_w0, A, h, ids, psis, buckets,
               kl_weight):
    """Gradients of head_loss with respect to W_lm, W_r and b_r."""
    n = len(A)
    G = logit_grads(lm_w, lm_w0, A, ids, kl_weight)
    X = np.concatenate([np.asarray(h, np.float64), psis], axis=1)
    S = X @ np.asarray(rank_w, np.float64).T + np.asarray(rank_b, np.float64)
    Q = np.exp(S - np.array([logsumexp(s) for s in S])[:, None])
    Q[np.arange(n), buckets] -= 1.0
    Q /= n
    return G.T @ A, Q.T @ X, Q.sum(axis=0)


def head_update(lm_w, rank_w, rank_b, lm_w0, h, targets, final_norm, eps,
                num: Numerics, lr, kl_weight, d2t=None):
    """One head-only step; returns (new LM head in float64 before storage
    rounding, new rank-head weight, new rank-head bias, loss before the
    step)."""
    A, ids, psis, buckets = prepare(lm_w, h, targets, final_norm, eps, num,
                                    d2t)
    loss = head_loss(lm_w, rank_w, rank_b, lm_w0, A, h, ids, psis, buckets,
                     kl_weight)
    gw, gr, gb = head_grads(lm_w, rank_w, rank_b, lm_w0, A, h, ids, psis,
                            buckets, kl_weight)
    return (np.asarray(lm_w, np.float64) - lr * gw,
            np.asarray(rank_w, np.float64) - lr * gr,
            np.asarray(rank_b, np.float64) - lr * gb, loss)
