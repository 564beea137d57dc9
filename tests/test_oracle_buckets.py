"""Forced rank-head buckets (the paper-frequency workload knob).

Random-init rank heads do not produce the bucket mix of a trained drafter,
so a workload may force each drafter row's bucket from seeded draws with the
class frequencies of the rank-head quality table (App. B).  Pins:
* the draws have those frequencies and are keyed per sequence;
* forcing changes only the bucket (and so the branching): a forced bucket
  equal to the rank head's own argmax reproduces the unforced iteration;
* the tree shapes that the forced buckets imply (all b0: a chain plus one
  sibling per row; all b3 with b(b3) = 0: no drafted node at all);
* out-of-range values clamp to 0..3;
* greedy acceptance stays lossless under forced buckets;
* the uniform fixed-k tree of the rank-guided-branching ablation (Sec. 4):
  all rows b1, every bucket branching k.
"""
import copy

import numpy as np
import pytest

import synth
from oracle import specdec
from oracle.model import Drafter, Target

SHAPE = synth.ModelShape(2, 64, 4, 2, 16, 96, 97)
BMAP = (2, 4, 10, 0)


def _wl(K=3, M=3, B_max=3, budget=40, plen=11):
    return synth.Workload("pin", "f32", SHAPE, 1, K=K, M=M, B_max=B_max,
                          budget=budget, n_seqs=1, prompt_len=(plen, plen),
                          branch_map=BMAP)


def _models(w, seed=0):
    tw = synth.make_weights(synth.target_specs(w.target), seed, w.dtype,
                            jitter=0.1)
    dw = synth.make_weights(synth.drafter_specs(w.target, w.drafter_layers,
                                                w.K), seed, w.dtype,
                            jitter=0.1)
    tgt = Target(tw, w.target, w.dtype, w.tap_layers)
    return tgt, Drafter(dw, w.target, w.dtype, w.drafter_layers, tgt.embed)


def test_draw_frequencies_and_keying():
    b = synth.paper_buckets(0, 0, 4, 200_000)
    assert b.dtype == np.int32 and b.min() >= 0 and b.max() <= 3
    freq = np.bincount(b.ravel(), minlength=4) / b.size
    want = np.array(synth.PAPER_BUCKET_PERMILLE) / 1000.0
    # binomial standard error at 8e5 draws is < 5e-4
    assert np.abs(freq - want).max() < 3e-3, freq
    # sequence s draws the same values whatever the batch size
    assert (synth.paper_buckets(0, 0, 2, 64)[1] ==
            synth.paper_buckets(0, 0, 5, 64)[1]).all()
    # iterations and seeds give different streams
    assert (synth.paper_buckets(0, 1, 1, 64) !=
            synth.paper_buckets(0, 0, 1, 64)).any()
    assert (synth.paper_buckets(1, 0, 1, 64) !=
            synth.paper_buckets(0, 0, 1, 64)).any()


def test_forcing_the_argmax_changes_nothing():
    w = _wl()
    tgt, dr = _models(w)
    st = specdec.prefill(tgt, dr, synth.prompts(w)[0])
    free = specdec.iteration(tgt, dr, copy.deepcopy(st), w)
    own = np.array([r.bucket for r in free["rows"]], np.int32)
    forced = specdec.iteration(tgt, dr, copy.deepcopy(st), w, buckets=own)
    assert [(n.token, n.parent, n.row, n.rank) for n in forced["tree"].nodes] \
        == [(n.token, n.parent, n.row, n.rank) for n in free["tree"].nodes]
    assert forced["committed"] == free["committed"]


def test_all_b0_rows_give_chain_plus_one_sibling():
    w = _wl(K=3, M=1, budget=40)
    tgt, dr = _models(w)
    st = specdec.prefill(tgt, dr, synth.prompts(w)[0])
    rec = specdec.iteration(tgt, dr, st, w,
                            buckets=np.zeros(w.rows_per_seq, np.int32))
    tree = rec["tree"]
    assert all(r.bucket == 0 and r.branch == BMAP[0] for r in rec["rows"])
    # b(b0) = 2: each of the K rows adds its rank-1 (chain) and rank-2 token
    assert len(tree) == 1 + 2 * w.K
    assert sorted(n.rank for n in tree.nodes[1:]) == [1] * w.K + [2] * w.K
    assert max(n.depth for n in tree.nodes) == w.K


def test_all_b3_rows_draft_nothing_and_clamp():
    w = _wl()
    tgt, dr = _models(w)
    st = specdec.prefill(tgt, dr, synth.prompts(w)[0])
    ref = specdec.iteration(tgt, dr, copy.deepcopy(st), w,
                            buckets=np.full(w.rows_per_seq, 3, np.int32))
    assert len(ref["tree"]) == 1 and ref["tau"] == 1
    assert all(r.bucket == 3 and r.branch == 0 for r in ref["rows"])
    # values above 3 clamp to b3, below 0 to b0
    hi = specdec.iteration(tgt, dr, copy.deepcopy(st), w,
                           buckets=np.full(w.rows_per_seq, 9, np.int32))
    assert len(hi["tree"]) == 1
    lo = specdec.iteration(tgt, dr, copy.deepcopy(st), w,
                           buckets=np.full(w.rows_per_seq, -5, np.int32))
    assert all(r.bucket == 0 for r in lo["rows"])


@pytest.mark.parametrize("seed", [0, 3])
def test_lossless_under_paper_buckets(seed):
    w = _wl()
    tgt, dr = _models(w, seed)
    prompt = synth.prompts(w)[0]
    ref = specdec.greedy_decode(tgt, prompt, 20)
    out, taus = specdec.speculative_decode(
        tgt, dr, prompt, w, 20,
        buckets=lambda i: synth.paper_buckets(seed, i, 1, w.rows_per_seq)[0])
    assert out == ref
    assert all(t >= 1 for t in taus)


def test_uniform_fixed_k_tree():
    """The rank-guided-branching ablation: every row contributes its top-k
    tokens under the same parent, and every sibling is a start candidate
    (chain end first, then siblings by cumulative log-probability)."""
    k = 3
    w = synth.uniform_tree(_wl(K=3, M=2, B_max=3, budget=60), k)
    assert w.branch_map == (k, k, k, k)
    tgt, dr = _models(w)
    st = specdec.prefill(tgt, dr, synth.prompts(w)[0])
    rec = specdec.iteration(tgt, dr, st, w,
                            buckets=synth.uniform_buckets(1, w.rows_per_seq)[0])
    tree, e1 = rec["tree"], rec["expansions"][0]
    assert e1["first_new"] == 1
    block1 = tree.nodes[1:1 + w.K * k]
    assert len(block1) == w.K * k
    for kk in range(w.K):
        sib = block1[kk * k:(kk + 1) * k]
        assert [n.rank for n in sib] == list(range(1, k + 1))
        assert len({n.parent for n in sib}) == 1
        assert sib[0].depth == kk + 1
    chain_end = 1 + (w.K - 1) * k
    sibs = [i for i in range(1, 1 + w.K * k) if tree.nodes[i].rank >= 2]
    by_cum = sorted(sibs, key=lambda i: (-tree.nodes[i].cum_logp, i))
    want = [chain_end] + by_cum[:w.B_max - 1]
    assert [sp.node for sp in rec["expansions"][1]["starts"]] == want
