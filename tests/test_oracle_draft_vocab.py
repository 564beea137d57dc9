"""Reduced drafter vocabulary (App. A: the drafter predicts over the most
frequent target tokens; its ids map to target ids).

Pins:
* restriction: a reduced drafter whose LM-head rows are the full drafter's
  rows at the mapped ids has, row by row, exactly the full drafter's logits
  at those ids, and its top-10 tokens are the brute-force top-10 of the full
  logits restricted to the mapped ids (a transposed or inverted map fails);
* every drafted token lies in the map's image;
* greedy acceptance stays lossless;
* the synthetic map is strictly increasing, in range and seeded.
"""
import copy
import dataclasses

import numpy as np
import pytest

import synth
from oracle import specdec
from oracle.model import Drafter, Target

SHAPE = synth.ModelShape(2, 64, 4, 2, 16, 96, 97)
VD = 40


def _wl(draft_vocab=VD, K=3, M=2, B_max=3, budget=30, plen=11):
    return synth.Workload("pin", "f32", SHAPE, 2, K=K, M=M, B_max=B_max,
                          budget=budget, n_seqs=1, prompt_len=(plen, plen),
                          draft_vocab=draft_vocab)


def _models(w, seed=0):
    tw = synth.make_weights(synth.target_specs(w.target), seed, w.dtype,
                            jitter=0.1)
    dw = synth.drafter_weights(w, seed, jitter=0.1)
    tgt = Target(tw, w.target, w.dtype, w.tap_layers)
    return tgt, Drafter(dw, w.target, w.dtype, w.drafter_layers, tgt.embed), dw


def test_map_properties():
    m = synth.draft_vocab_map(0, 128256, 32000)
    assert m.dtype == np.int32 and len(m) == 32000
    assert (np.diff(m) > 0).all() and m[0] >= 0 and m[-1] < 128256
    assert (m == synth.draft_vocab_map(0, 128256, 32000)).all()
    assert (m != synth.draft_vocab_map(1, 128256, 32000)).any()


def test_restriction_of_the_full_drafter():
    wf = _wl(draft_vocab=0)
    tgt, full, raw = _models(wf)
    d2t = synth.draft_vocab_map(3, SHAPE.vocab, VD)
    red_raw = dict(raw)
    red_raw["d.lm_head"] = raw["d.lm_head"][d2t]
    red_raw["d.d2t"] = d2t
    red = Drafter(red_raw, wf.target, wf.dtype, wf.drafter_layers, tgt.embed)
    st = specdec.prefill(tgt, full, synth.prompts(wf)[0])
    a = specdec.iteration(tgt, full, copy.deepcopy(st), wf)
    rows_f = a["rows"]
    # the same block-1 rows through the reduced drafter
    st2 = copy.deepcopy(st)
    tree = specdec.DraftTree(st2.root, wf.budget)
    rows = []
    seg = red.new_segment(wf.rows_per_seq)
    starts = [specdec.Start(0, st2.root, st2.T,
                            red.cond_from_taps(st2.cond_taps), [])]
    specdec.expand_block(red, st2, tree, rows, seg, starts, wf.K, 1,
                         wf.branch_map)
    assert len(rows) == wf.K
    for rf, rr in zip(rows_f[:wf.K], rows):
        # block 1 depends only on the start, not on the vocabulary: the
        # hidden states agree, and the logits are the restriction
        assert np.allclose(rr.h_last, rf.h_last, rtol=0, atol=1e-12)
        assert rr.logits.shape == (VD,)
        assert np.allclose(rr.logits, rf.logits[d2t], rtol=0, atol=1e-12)
        z = rf.logits[d2t]
        brute = d2t[np.lexsort((d2t, -z))[:10]]
        assert list(rr.topk) == list(brute)
        assert list(red.to_target(rr.topk_d)) == list(rr.topk)


@pytest.mark.parametrize("seed", [0, 2])
def test_drafted_tokens_in_map_and_lossless(seed):
    w = _wl()
    tgt, dr, raw = _models(w, seed)
    image = set(raw["d.d2t"].tolist())
    st = specdec.prefill(tgt, dr, synth.prompts(w)[0])
    for _ in range(3):
        rec = specdec.iteration(tgt, dr, st, w)
        assert all(n.token in image for n in rec["tree"].nodes[1:])
        for r in rec["rows"]:
            assert len(r.logits) == VD
            assert abs(r.lse - np.logaddexp.reduce(r.logits)) < 1e-9
    prompt = synth.prompts(w)[0]
    ref = specdec.greedy_decode(tgt, prompt, 16)
    out, _ = specdec.speculative_decode(tgt, dr, prompt, w, 16)
    assert out == ref


def test_paper_shaped_drafter_workload():
    w = synth.WORKLOADS["llama3-8b-paper-drafter"]
    assert w.drafter_layers == 2 and w.draft_vocab == 32000
    assert (w.K, w.M, w.budget, w.n_seqs) == (4, 2, 60, 1)
    assert dataclasses.replace(w, draft_vocab=0).draft_vocab == 0
