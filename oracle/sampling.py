"""Stochastic tree verification at temperature T > 0 (oracle).

Test infrastructure: see the package docstring.

The paper evaluates SpecBlock at temperature 1.0 as well as greedily (Sec. 4
setup and main results), verifying the draft tree by rejection sampling,
but does not spell the algorithm out.  This is the standard lossless
multi-candidate scheme (speculative sampling, Leviathan et al. 2023, applied
recursively over a node's children as in SpecInfer, Miao et al. 2024) with
one twist that the tree construction imposes: the children of a node are
the drafter's *deterministic* top-b tokens, so each child is tested as a
point-mass draft against the current residual distribution.

At node n with target distribution p_n = softmax(z_n / T):
* the children are tested in increasing node id; a child whose token was
  already rejected at n has residual probability zero and is skipped
  without a draw;
* child c (token x) is accepted when u_acc[c] < r(x), where r is the
  residual distribution: p_n with the rejected tokens removed and
  renormalised.  Accepting moves the walk to c (whose own children are
  tested against p_c); rejecting removes x from the residual;
* when no child is accepted the bonus token is drawn from the residual by
  inverse transform in increasing token id: the smallest x whose cumulative
  residual mass exceeds u_bonus[n] times the residual total.

Each test is a speculative-sampling step with draft q = delta_x, accepting
with probability min(1, r(x) / q(x)) = r(x) and otherwise continuing with
the renormalised positive part of r - q, which is r without x; so the token
emitted at every node is distributed exactly as p_n, whatever the tree.

Readings (ours; parity of the order of tests and of the inverse-transform
direction is unpinned by the paper): children in node-id order; one uniform
per child test indexed by the child's node id, one per bonus draw indexed by
the node where the walk stops.
"""
from __future__ import annotations

import numpy as np

from .tree import DraftTree


def target_probs(z, temperature: float) -> np.ndarray:
    """softmax(z / T) in float64."""
    x = np.asarray(z, dtype=np.float64) / float(temperature)
    x = x - x.max()
    e = np.exp(x)
    return e / e.sum()


def accept_sample(tree: DraftTree, logits, temperature: float, u_acc,
                  u_bonus) -> dict:
    """Stochastic acceptance walk over ``tree``.

    logits[n] are the target logits at node n (the distribution of the token
    after node n's); u_acc and u_bonus are uniforms in [0, 1) indexed by node
    id.  Returns the accepted node ids (root excluded), the bonus token and
    the smallest margins of the discrete decisions (|u - r(x)| over the tests
    made, and the distance of the bonus target from the neighbouring
    cumulative-mass boundaries, both relative to the residual total), which
    tests use to decide where a lower-precision run must agree exactly."""
    if not temperature > 0:
        raise ValueError("temperature must be positive")
    cur, path = 0, []
    test_margin = np.inf
    while True:
        p = target_probs(logits[cur], temperature)
        rejected: list = []
        mass = 1.0
        moved = False
        for c in sorted(tree.children(cur)):
            x = tree.nodes[c].token
            if x in rejected:
                continue
            r = p[x] / mass
            test_margin = min(test_margin, abs(float(u_acc[c]) - r))
            if u_acc[c] < r:
                path.append(c)
                cur = c
                moved = True
                break
            rejected.append(x)
            mass -= p[x]
        if not moved:
            break
    # bonus: inverse transform over the residual at the last node
    w = p.copy()
    w[rejected] = 0.0
    cdf = np.cumsum(w)
    total = cdf[-1]
    target = float(u_bonus[cur]) * total
    bonus = int(np.searchsorted(cdf, target, side="right"))
    bonus = min(bonus, len(w) - 1)
    while w[bonus] == 0.0 and bonus > 0:      # never a removed token
        bonus -= 1
    lo = cdf[bonus - 1] if bonus > 0 else 0.0
    cdf_margin = min(target - lo, cdf[bonus] - target) / total
    return dict(path=path, bonus=bonus, test_margin=test_margin,
                cdf_margin=cdf_margin)
