"""Pins of stochastic tree verification (temperature T > 0).

Lossless means: the token emitted at every node of the walk is distributed
as the target's p_n at that node, whatever the draft tree.  Checked
empirically on small synthetic trees (Monte Carlo with many uniforms, against
the target probabilities within a few standard errors), including duplicate
child tokens and nodes without children; and in the deterministic limit,
where a one-hot target must reproduce greedy acceptance exactly, and a
near-zero temperature speculative decode must reproduce the target's greedy
decode (losslessness).
"""
import numpy as np
import pytest

import synth
from oracle import specdec
from oracle.model import Drafter, Target
from oracle.sampling import accept_sample, target_probs
from oracle.tree import DraftTree, accept

V = 6


def _tree():
    """root -> a(2) b(4) c(2, duplicate of a) d(5); a -> e(1) f(3); d -> g(0)."""
    t = DraftTree(0, 16)
    a = t.add(2, 0, 0, 1, 0.0)
    b = t.add(4, 0, 0, 2, 0.0)
    c = t.add(2, 0, 1, 1, 0.0)
    d = t.add(5, 0, 1, 2, 0.0)
    e = t.add(1, a, 2, 1, 0.0)
    f = t.add(3, a, 2, 2, 0.0)
    g = t.add(0, d, 3, 1, 0.0)
    return t, dict(a=a, b=b, c=c, d=d, e=e, f=f, g=g)


def _logits(t, ids, rng):
    z = rng.standard_normal((len(t), V)) * 1.5
    z[ids["c"]] = z[ids["a"]]          # same context, same target distribution
    return z


@pytest.mark.parametrize("temperature", [1.0, 0.7])
def test_emitted_tokens_follow_the_target(temperature):
    rng = np.random.default_rng(5)
    t, ids = _tree()
    z = _logits(t, ids, rng)
    N = 60_000
    ua = rng.random((N, len(t)))
    ub = rng.random((N, len(t)))
    first = np.zeros(V)
    second = {n: np.zeros(V) for n in (ids["a"], ids["d"])}
    for i in range(N):
        r = accept_sample(t, z, temperature, ua[i], ub[i])
        toks = [t.nodes[n].token for n in r["path"]] + [r["bonus"]]
        first[toks[0]] += 1
        if r["path"] and r["path"][0] in second:
            second[r["path"][0]][toks[1]] += 1
        # invariant: a path of parent -> child edges
        prev = 0
        for n in r["path"]:
            assert t.nodes[n].parent == prev
            prev = n
    p0 = target_probs(z[0], temperature)
    se = np.sqrt(p0 * (1 - p0) / N)
    assert np.all(np.abs(first / N - p0) < 5 * se + 1e-4), (first / N, p0)
    for n, cnt in second.items():
        m = cnt.sum()
        assert m > 2000
        pn = target_probs(z[n], temperature)
        se = np.sqrt(pn * (1 - pn) / m)
        assert np.all(np.abs(cnt / m - pn) < 5 * se + 1e-4), (n, cnt / m, pn)


def test_no_children_is_a_plain_draw():
    rng = np.random.default_rng(1)
    t = DraftTree(0, 4)
    z = rng.standard_normal((1, V))
    N = 40_000
    cnt = np.zeros(V)
    for u in rng.random(N):
        r = accept_sample(t, z, 1.0, [0.0], [u])
        assert r["path"] == []
        cnt[r["bonus"]] += 1
    p = target_probs(z[0], 1.0)
    assert np.all(np.abs(cnt / N - p) < 5 * np.sqrt(p * (1 - p) / N) + 1e-4)


def test_one_hot_target_is_greedy_acceptance():
    rng = np.random.default_rng(2)
    t, ids = _tree()
    for trial in range(200):
        z = rng.standard_normal((len(t), V))
        z[ids["c"]] = z[ids["a"]]
        # make the target's choice often a child token
        for n in range(len(t)):
            kids = t.children(n)
            if kids and rng.random() < 0.7:
                z[n, t.nodes[int(rng.choice(kids))].token] += 3.0
        zz = z * 1e4                      # softmax is one-hot in float64
        greedy = np.array([int(np.argmax(r)) for r in z])
        path, bonus = accept(t, greedy)
        r = accept_sample(t, zz, 1.0, rng.random(len(t)) * 0.999,
                          rng.random(len(t)))
        assert r["path"] == path and r["bonus"] == bonus, trial


SHAPE = synth.ModelShape(2, 64, 4, 2, 16, 96, 97)


def test_near_zero_temperature_decode_is_lossless():
    w = synth.Workload("pin", "f32", SHAPE, 1, K=3, M=2, B_max=3, budget=24,
                       n_seqs=1, prompt_len=(11, 11))
    tw = synth.make_weights(synth.target_specs(w.target), 0, w.dtype,
                            jitter=0.1)
    dw = synth.drafter_weights(w, 0, jitter=0.1)
    tgt = Target(tw, w.target, w.dtype, w.tap_layers)
    dr = Drafter(dw, w.target, w.dtype, w.drafter_layers, tgt.embed)
    prompt = synth.prompts(w)[0]
    ref = specdec.greedy_decode(tgt, prompt, 16)
    rng = np.random.default_rng(9)

    def sampling(i):
        return (1e-6, rng.random(w.budget), rng.random(w.budget))
    out, _ = specdec.speculative_decode(tgt, dr, prompt, w, 16,
                                        sampling=sampling)
    assert out == ref


def test_rejects_nonpositive_temperature():
    t = DraftTree(0, 2)
    with pytest.raises(ValueError):
        accept_sample(t, np.zeros((1, V)), 0.0, [0.5], [0.5])
