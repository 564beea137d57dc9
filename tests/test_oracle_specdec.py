"""Pins of the whole iteration: losslessness and cache bookkeeping.

Losslessness: greedy draft-then-verify commits exactly the target's own
greedy decode, whatever the drafter proposes.
Random-init drafters rarely match, so trees are also *planted*: after
drafting, a root path is rewritten with the target's greedy continuation,
which must then be accepted exactly (tau = planted depth + 1).
"""
import numpy as np
import pytest

import synth
from oracle import specdec
from oracle.model import Drafter, Target

SHAPE = synth.ModelShape(2, 64, 4, 2, 16, 96, 97)


def _wl(K=3, M=3, B_max=3, budget=24, plen=11):
    return synth.Workload("pin", "f32", SHAPE, 1, K=K, M=M, B_max=B_max,
                          budget=budget, n_seqs=1, prompt_len=(plen, plen))


def _models(w, seed=0):
    tw = synth.make_weights(synth.target_specs(w.target), seed, w.dtype,
                            jitter=0.1)
    dw = synth.make_weights(synth.drafter_specs(w.target, w.drafter_layers,
                                                w.K), seed, w.dtype,
                            jitter=0.1)
    tgt = Target(tw, w.target, w.dtype, w.tap_layers)
    return tgt, Drafter(dw, w.target, w.dtype, w.drafter_layers, tgt.embed)


@pytest.mark.parametrize("bmap", [(2, 4, 10, 0), (2, 4, 6, 4)])
def test_lossless_random_drafter(bmap):
    w = _wl()
    tgt, dr = _models(w)
    prompt = synth.prompts(w)[0]
    ref = specdec.greedy_decode(tgt, prompt, 20)
    out, taus = specdec.speculative_decode(tgt, dr, prompt, w, 20, bmap)
    assert out == ref
    assert all(t >= 1 for t in taus)


def _planter(ref_stream, st_holder, rng, depths, log):
    """Rewrite a random root-to-node path with the greedy continuation."""
    def plant(tree, rows):
        st = st_holder[0]
        done = len(st.tokens) - st_holder[1]       # committed since prefill
        want = depths[len(log) % len(depths)]
        cands = [i for i in range(1, len(tree)) if tree.nodes[i].depth ==
                 min(want, max(n.depth for n in tree.nodes))]
        leaf = int(rng.choice(cands))
        path = tree.anc_or_self(leaf)[1:]
        for j, n in enumerate(path):
            tok = ref_stream[done + j]
            p = tree.nodes[n].parent
            for c in tree.children(p):          # keep children distinct
                if c != n and tree.nodes[c].token == tok:
                    tree.nodes[c].token = (tok + 1) % SHAPE.vocab
            tree.nodes[n].token = tok
        log.append(len(path))
    return plant


@pytest.mark.parametrize("seed", [0, 1])
def test_lossless_planted_trees(seed):
    w = _wl(K=3, M=3, B_max=3, budget=24)
    tgt, dr = _models(w, seed)
    prompt = synth.prompts(w, seed=seed + 10)[0]
    n_new = 40
    ref = specdec.greedy_decode(tgt, prompt, n_new + 12)
    st = specdec.prefill(tgt, dr, prompt)
    holder = [st, len(st.tokens)]
    rng = np.random.default_rng(seed)
    log = []
    plant = _planter(ref[1:], holder, rng, [1, 2, 3, 4, 5, 6, 7], log)
    out = [st.root]
    fallbacks = 0
    while len(out) < n_new:
        rec = specdec.iteration(tgt, dr, st, w, None, plant)
        # the planted path is accepted exactly (a random extra match would
        # need a drafted token to equal the target's choice, prob ~ 1/V)
        assert rec["tau"] >= log[-1] + 1
        out += rec["committed"]
        fallbacks += rec["fallback"]
    assert out[:n_new] == ref[:n_new]
    assert max(log) > w.K       # a planted path crossed a block boundary
    assert fallbacks > 0          # the catch-up path was exercised
    # target cache == a causal pass over the committed stream
    toks = st.tokens[:-1]
    n = len(toks)
    seg = tgt.new_segment(n)
    idx = np.arange(n)
    tgt.forward(toks, idx, idx, [list(range(r + 1)) for r in idx],
                tgt.new_prefix(), seg)
    assert len(st.tkv) == n == st.T
    for layer in range(SHAPE.n_layers):
        np.testing.assert_allclose(st.tkv.k[layer], seg.k[layer], rtol=1e-10,
                                   atol=1e-10)
        np.testing.assert_allclose(st.tkv.v[layer], seg.v[layer], rtol=1e-10,
                                   atol=1e-10)
    assert len(st.dkv) == st.T


def test_bonus_entry_reuse_equals_catch_up():
    """With nothing accepted, the drafter entry for the bonus position is
    block-1 row 1, which must equal a K = 1 catch-up row from the root."""
    w = _wl()
    tgt, dr = _models(w)
    st = specdec.prefill(tgt, dr, synth.prompts(w)[0])
    T, root, taps = st.T, st.root, st.cond_taps.copy()
    before = dr.new_prefix()
    for layer in range(1):
        before.k[layer] = st.dkv.k[layer].copy()
        before.v[layer] = st.dkv.v[layer].copy()
    rec = specdec.iteration(tgt, dr, st, w)
    if rec["tau"] != 1:
        pytest.skip("random drafter matched the target")
    seg = specdec.catch_up(dr, dr.cond_from_taps(taps)[None], [root], T,
                           before)
    np.testing.assert_allclose(st.dkv.k[0][T], seg.k[0][0], rtol=1e-12,
                               atol=1e-12)
    np.testing.assert_allclose(st.dkv.v[0][T], seg.v[0][0], rtol=1e-12,
                               atol=1e-12)


def test_depth_and_forward_count_bounds():
    """At most M drafter forwards per iteration and depth <= M*K."""
    w = _wl(K=2, M=3, B_max=2, budget=30)
    tgt, dr = _models(w)
    st = specdec.prefill(tgt, dr, synth.prompts(w)[0])
    for _ in range(3):
        rec = specdec.iteration(tgt, dr, st, w, (1, 1, 1, 1))
        assert len(rec["expansions"]) <= w.M
        assert max(n.depth for n in rec["tree"].nodes) <= w.M * w.K
    # with b = 1 everywhere and room in the budget, the chain reaches M*K
    assert max(n.depth for n in rec["tree"].nodes) == w.M * w.K
