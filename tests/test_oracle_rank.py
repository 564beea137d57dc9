"""Pins of psi, the rank-to-bucket rule and the branching maps."""
import os

import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

from oracle.rank import (BRANCH_MAP_CONCENTRATE, BRANCH_MAP_FALLBACK,
                         bucket_of_rank, bucket_of_scores, psi, topk_ids)

HERE = os.path.dirname(__file__)


def _golden():
    rule, maps = {}, []
    with open(os.path.join(HERE, "golden", "rank_rules.txt")) as f:
        for line in f:
            a = line.split()
            if not a or a[0].startswith("#"):
                continue
            if a[0] == "rank_to_bucket":
                for kv in a[1:]:
                    r, b = kv.split(":")
                    rule[int(r)] = int(b)
            elif a[0] == "branch_map":
                maps.append(tuple(int(x) for x in a[1:]))
    return rule, maps


def test_rank_rule_and_maps_match_paper_text():
    rule, maps = _golden()
    for r, b in rule.items():
        assert bucket_of_rank(r) == b
    assert maps == [BRANCH_MAP_CONCENTRATE, BRANCH_MAP_FALLBACK]


@pytest.mark.parametrize("V", [16, 1024, 128256])
def test_psi_uniform_closed_form(V):
    p = psi(np.full(V, 0.37))
    np.testing.assert_allclose(p[:10], -np.log(V), rtol=1e-12)
    np.testing.assert_allclose(p[10:13], 0.0, atol=0)
    np.testing.assert_allclose(p[13], 1.0 / V, rtol=1e-12)
    np.testing.assert_allclose(p[14], np.log(V), rtol=1e-12)


def test_psi_two_level_closed_form():
    """Top token at logit a, the V-1 others at 0."""
    V, a = 1000, 5.0
    z = np.zeros(V)
    z[123] = a
    Z = np.exp(a) + V - 1
    p1 = np.exp(a) / Z
    q = 1 / Z
    p = psi(z)
    assert p[0] == pytest.approx(np.log(p1), rel=1e-12)
    np.testing.assert_allclose(p[1:10], np.log(q), rtol=1e-12)
    np.testing.assert_allclose(p[10:13], a, rtol=1e-12)
    assert p[13] == pytest.approx(p1, rel=1e-12)
    H = -(p1 * np.log(p1) + (V - 1) * q * np.log(q))
    assert p[14] == pytest.approx(H, rel=1e-12)


def test_psi_matches_library_on_random_logits():
    rng = np.random.default_rng(4)
    z = rng.standard_normal(5000) * 1.3
    p = psi(z)
    tv, _ = torch.topk(torch.tensor(z), 10)
    lse = scipy.special.logsumexp(z)
    np.testing.assert_allclose(p[:10], tv.numpy() - lse, rtol=1e-12)
    srt = np.sort(z)[::-1]
    np.testing.assert_allclose(p[10:13], [srt[0] - srt[1], srt[0] - srt[2],
                                          srt[0] - srt[4]], rtol=1e-12)
    assert p[13] == pytest.approx(np.exp(srt[0] - lse), rel=1e-12)
    ent = scipy.stats.entropy(scipy.special.softmax(z))
    assert p[14] == pytest.approx(ent, rel=1e-11)


def test_topk_order_and_ties():
    z = np.array([1.0, 3.0, 3.0, -1.0, 3.0, 2.0])
    np.testing.assert_array_equal(topk_ids(z, 5), [1, 2, 4, 5, 0])
    rng = np.random.default_rng(5)
    z = rng.standard_normal(777)
    np.testing.assert_array_equal(topk_ids(z, 10),
                                  torch.topk(torch.tensor(z), 10)[1].numpy())


def test_bucket_argmax_ties_low():
    assert bucket_of_scores([0.5, 2.0, 2.0, 1.0]) == 1
    assert bucket_of_scores([3.0, 3.0, 3.0, 3.0]) == 0
    assert bucket_of_scores([-1, -2, -0.5, -0.5]) == 2


# --- rank head g_phi over [h^(L), psi] (Eq. 4) ---------------------------
# Crafted heads that read one block of the input at a time: a swapped
# concatenation [psi, h], a dropped block or a dropped bias each change the
# winning bucket or the score value below.

def _rank_case():
    d = 8
    h = np.array([0.5, -1.0, 2.0, 7.0, -3.0, 0.25, 1.5, -0.75])
    # two-level logits: top token at 5, the other 999 at 0 (closed-form psi)
    z = np.zeros(1000)
    z[7] = 5.0
    Z = np.exp(5.0) + 999.0
    p1 = np.exp(5.0) / Z
    return d, h, psi(z), p1


def test_rank_head_reads_h_block_first():
    from oracle.rank import rank_scores
    d, h, ps, _ = _rank_case()
    w = np.zeros((4, d + 15))
    w[1, 3] = 1.0          # bucket b1 scores h^(L)[3] = 7
    w[2, 4] = 1.0          # bucket b2 scores h^(L)[4] = -3
    s = rank_scores(w, np.zeros(4), h, ps)
    np.testing.assert_array_equal(s, [0.0, 7.0, -3.0, 0.0])
    assert bucket_of_scores(s) == 1


def test_rank_head_reads_psi_block_after_h():
    from oracle.rank import rank_scores
    d, h, ps, p1 = _rank_case()
    w = np.zeros((4, d + 15))
    w[2, d + 13] = 10.0    # psi[13] = top-1 probability
    w[3, d + 10] = -1.0    # psi[10] = z1 - z2 = 5 (two-level logits)
    s = rank_scores(w, np.zeros(4), h, ps)
    assert s[0] == 0.0 and s[1] == 0.0
    assert s[2] == pytest.approx(10.0 * p1, rel=1e-12)
    assert s[3] == pytest.approx(-5.0, rel=1e-12)
    assert bucket_of_scores(s) == 2


def test_rank_head_adds_bias():
    from oracle.rank import rank_scores
    d, h, ps, _ = _rank_case()
    b = np.array([0.0, -1.0, 0.5, 2.0])
    s = rank_scores(np.zeros((4, d + 15)), b, h, ps)
    np.testing.assert_array_equal(s, b)
    assert bucket_of_scores(s) == 3
    # bias and one weight together: b0 wins with 1 + h[0] = 1.5
    w = np.zeros((4, d + 15))
    w[0, 0] = 1.0
    s = rank_scores(w, np.array([1.0, 0.0, 0.0, 1.4]), h, ps)
    np.testing.assert_allclose(s, [1.5, 0.0, 0.0, 1.4], rtol=1e-15)
    assert bucket_of_scores(s) == 0
