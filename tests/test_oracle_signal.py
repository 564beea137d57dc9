"""Pins of the verifier-derived update signal (Sec. 3.4, Eq. 8).

r is the drafter's probability of the target's token at the rejected
position, read from the drafter row that predicted that position.
* When the root's position is rejected (nothing accepted), that row is the
  first row of block 1; a block's first row is one autoregressive drafter
  step (the drafter forward reduces to one, see test_oracle_drafter), so r
  must equal the probability that a K = 1
  block started at the root assigns to the bonus token.
* r is None exactly when no drafter row continues the last accepted node
  (the commit then needs a catch-up row), and lies in [0, 1] otherwise.
* With a reduced drafter vocabulary, r = 0 exactly when the bonus token is
  outside it.
"""
import copy
import dataclasses

import numpy as np
import pytest

import synth
from oracle import specdec
from oracle.model import Drafter, Target
from oracle.numerics import logsumexp

SHAPE = synth.ModelShape(2, 64, 4, 2, 16, 96, 97)


def _setup(draft_vocab=0, seed=0, K=3):
    w = synth.Workload("pin", "f32", SHAPE, 1, K=K, M=2, B_max=3, budget=30,
                       n_seqs=1, prompt_len=(11, 11), draft_vocab=draft_vocab)
    tw = synth.make_weights(synth.target_specs(w.target), seed, w.dtype,
                            jitter=0.1)
    dw = synth.drafter_weights(w, seed, jitter=0.1)
    tgt = Target(tw, w.target, w.dtype, w.tap_layers)
    dr = Drafter(dw, w.target, w.dtype, w.drafter_layers, tgt.embed)
    st = specdec.prefill(tgt, dr, synth.prompts(w)[0])
    return w, tgt, dr, st


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_root_rejection_is_one_drafter_step(seed):
    w, tgt, dr, st = _setup(seed=seed)
    rec = specdec.iteration(tgt, dr, copy.deepcopy(st), w)
    if rec["path"]:
        pytest.skip("random drafter matched the target")
    # a K = 1 block at the root, from scratch
    w1 = dataclasses.replace(w, K=1)
    s1 = copy.deepcopy(st)
    tree = specdec.DraftTree(s1.root, w.budget)
    rows = []
    seg = dr.new_segment(w1.rows_per_seq)
    start = specdec.Start(0, s1.root, s1.T, dr.cond_from_taps(s1.cond_taps),
                          [])
    specdec.expand_block(dr, s1, tree, rows, seg, [start], 1, 1,
                         w.branch_map)
    z = rows[0].logits
    want = float(np.exp(z[rec["bonus"]] - logsumexp(z)))
    assert rec["r_reject"] == pytest.approx(want, rel=1e-9, abs=1e-300)


def test_none_exactly_when_commit_needs_a_catch_up_row():
    for seed in range(4):
        w, tgt, dr, st = _setup(seed=seed, K=2)
        for _ in range(3):
            rec = specdec.iteration(tgt, dr, st, w)
            r = rec["r_reject"]
            assert (r is None) == rec["fallback"]
            if r is not None:
                assert 0.0 <= r <= 1.0


def test_reduced_vocabulary_zero_outside():
    seen_zero = seen_pos = 0
    for seed in range(6):
        w, tgt, dr, st = _setup(draft_vocab=32, seed=seed)
        image = set(dr.d2t.tolist())
        for _ in range(3):
            rec = specdec.iteration(tgt, dr, st, w)
            r = rec["r_reject"]
            if r is None:
                continue
            if rec["bonus"] in image:
                assert r > 0.0
                seen_pos += 1
            else:
                assert r == 0.0
                seen_zero += 1
    assert seen_zero and seen_pos
