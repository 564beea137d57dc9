"""Pins of the head-only drafter update (Sec. 3.4, App. A.3).

* The analytic gradients match central finite differences of the loss
  (LM head, rank-head weight and bias), with and without the KL term.
* A small step lowers the loss.
* With the training copy equal to the pre-deployment head the KL term and
  its gradient vanish: the step does not depend on lambda.
* A target outside a reduced vocabulary has no cross-entropy term and the
  give-up bucket b3 as its rank label.
* The target's rank agrees with a brute-force sort (larger logit first,
  equal logits by smaller id).
"""
import numpy as np
import pytest

from oracle.adapt import (drafter_id, head_grads, head_loss, head_update,
                          prepare, target_rank)
from oracle.numerics import Numerics

D, VD, N = 16, 23, 4


def _case(seed=0, d2t=None):
    rng = np.random.default_rng(seed)
    lm = rng.standard_normal((VD, D)) * 0.5
    lm0 = lm + rng.standard_normal((VD, D)) * 0.1
    rw = rng.standard_normal((4, D + 15)) * 0.3
    rb = rng.standard_normal(4) * 0.1
    h = rng.standard_normal((N, D))
    g = 1.0 + 0.1 * rng.standard_normal(D)
    vocab = VD if d2t is None else int(d2t[-1]) + 5
    tgt = rng.integers(0, vocab, size=N)
    return lm, lm0, rw, rb, h, g, tgt


@pytest.mark.parametrize("kl", [0.0, 0.7])
def test_gradients_match_finite_differences(kl):
    lm, lm0, rw, rb, h, g, tgt = _case(1)
    num = Numerics("f32")
    A, ids, psis, bk = prepare(lm, h, tgt, g, 1e-5, num)
    args = (A, h, ids, psis, bk, kl)
    gw, gr, gb = head_grads(lm, rw, rb, lm0, *args)
    eps = 1e-6
    rng = np.random.default_rng(3)
    for _ in range(12):
        v, k = rng.integers(VD), rng.integers(D)
        up, dn = lm.copy(), lm.copy()
        up[v, k] += eps
        dn[v, k] -= eps
        fd = (head_loss(up, rw, rb, lm0, *args) -
              head_loss(dn, rw, rb, lm0, *args)) / (2 * eps)
        assert fd == pytest.approx(gw[v, k], rel=1e-5, abs=1e-8)
    for _ in range(8):
        b, j = rng.integers(4), rng.integers(D + 15)
        up, dn = rw.copy(), rw.copy()
        up[b, j] += eps
        dn[b, j] -= eps
        fd = (head_loss(lm, up, rb, lm0, *args) -
              head_loss(lm, dn, rb, lm0, *args)) / (2 * eps)
        assert fd == pytest.approx(gr[b, j], rel=1e-5, abs=1e-8)
    for b in range(4):
        up, dn = rb.copy(), rb.copy()
        up[b] += eps
        dn[b] -= eps
        fd = (head_loss(lm, rw, up, lm0, *args) -
              head_loss(lm, rw, dn, lm0, *args)) / (2 * eps)
        assert fd == pytest.approx(gb[b], rel=1e-5, abs=1e-8)


def test_small_step_lowers_the_loss():
    lm, lm0, rw, rb, h, g, tgt = _case(2)
    num = Numerics("f32")
    A, ids, psis, bk = prepare(lm, h, tgt, g, 1e-5, num)
    nl, nr, nb, loss = head_update(lm, rw, rb, lm0, h, tgt, g, 1e-5, num,
                                   lr=0.05, kl_weight=0.3)
    after = head_loss(nl, nr, nb, lm0, A, h, ids, psis, bk, 0.3)
    assert after < loss


def test_kl_vanishes_at_the_pre_deployment_head():
    lm, _, rw, rb, h, g, tgt = _case(4)
    num = Numerics("f32")
    a = head_update(lm, rw, rb, lm, h, tgt, g, 1e-5, num, 0.1, 0.0)
    b = head_update(lm, rw, rb, lm, h, tgt, g, 1e-5, num, 0.1, 2.0)
    for x, y in zip(a[:3], b[:3]):
        assert np.allclose(x, y, rtol=0, atol=1e-14)


def test_out_of_vocabulary_target():
    d2t = np.array([1, 4, 5, 9, 11, 12, 20, 21, 30, 31, 33, 40, 41, 43, 50,
                    51, 52, 60, 61, 62, 70, 71, 80])
    assert len(d2t) == VD
    lm, _, rw, rb, h, g, _ = _case(5)
    tgt = np.array([2, 3, 6, 7])                  # none in the map
    assert all(drafter_id(d2t, y) is None for y in tgt)
    num = Numerics("f32")
    A, ids, psis, bk = prepare(lm, h, tgt, g, 1e-5, num, d2t)
    assert list(bk) == [3, 3, 3, 3]
    gw, _, _ = head_grads(lm, rw, rb, lm, A, h, ids, psis, bk, 1.0)
    assert np.abs(gw).max() < 1e-14               # no CE, no KL at theta_0


def test_target_rank_brute_force():
    rng = np.random.default_rng(6)
    for _ in range(50):
        z = np.round(rng.standard_normal(30), 1)   # ties happen
        i = int(rng.integers(30))
        order = sorted(range(30), key=lambda j: (-z[j], j))
        assert target_rank(z, i) == order.index(i) + 1


def test_drift_term_is_kl_of_training_head_from_pre_deployment_head():
    """Sec. 3.4's drift penalty is lambda KL(p_theta || p_theta0): on three
    tokens with p = (0.7, 0.2, 0.1) and p0 = (0.2, 0.3, 0.5) the two
    directions differ (0.6349 vs 0.6758) and the loss must carry the first.
    The cross-entropy terms are switched off (no target id) and the rank
    head scores all zero, which leaves its cross-entropy at log 4."""
    import scipy.stats
    p = np.array([0.7, 0.2, 0.1])
    p0 = np.array([0.2, 0.3, 0.5])
    lm = np.log(p)[:, None]            # d = 1, operand a = 1: z = log p
    lm0 = np.log(p0)[:, None]
    A = np.ones((1, 1))
    h = np.zeros((1, 1))
    psis = np.zeros((1, 15))
    rw, rb = np.zeros((4, 16)), np.zeros(4)
    lam = 2.0
    loss = head_loss(lm, rw, rb, lm0, A, h, [None], psis, np.array([0]), lam)
    fwd = scipy.stats.entropy(p, p0)   # KL(p || p0)
    rev = scipy.stats.entropy(p0, p)
    assert abs(fwd - rev) > 0.04
    assert fwd == pytest.approx(0.634897, abs=1e-6)
    assert loss == pytest.approx(lam * fwd + np.log(4.0), rel=1e-12)
    assert abs(loss - (lam * rev + np.log(4.0))) > 0.08
