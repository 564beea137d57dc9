"""Pins of the oracle's drafter block forward.

* the attention pattern and position ids of the paper's worked example
  (App. A.2 figure, golden fixture);
* block 1 on top of the catch-up prefix, and a block-2 expansion started
  from B_{1,1}, equal a causal run of transformers' Llama layer over the
  path's shifted inputs (brute force over the path; with K = 1 this is one
  autoregressive drafter step);
* invariants that follow from causal attention and the left-only shift:
  prefix consistency, causality in k, start-permutation invariance;
* later blocks bypass W_cond and carry the cached h^(L).
"""
import os

import numpy as np
import pytest
import torch

import synth
from oracle import specdec
from oracle.model import Drafter, Target
from oracle.tree import DraftTree

from hfref import drafter_trunk, layer_outputs, target_model

HERE = os.path.dirname(__file__)
SHAPE = synth.ModelShape(2, 64, 4, 2, 16, 96, 211)
W = synth.Workload("pin", "f32", SHAPE, 1, K=4, M=2, B_max=3, budget=40,
                   n_seqs=1, prompt_len=(9, 9))


def _models(w=W, seed=0):
    tw = synth.make_weights(synth.target_specs(w.target), seed, w.dtype,
                            jitter=0.1)
    dw = synth.make_weights(synth.drafter_specs(w.target, w.drafter_layers,
                                                w.K), seed, w.dtype,
                            jitter=0.1)
    tgt = Target(tw, w.target, w.dtype, w.tap_layers)
    dr = Drafter(dw, w.target, w.dtype, w.drafter_layers, tgt.embed)
    return tw, dw, tgt, dr


def _read_golden():
    rows, pos = [], None
    with open(os.path.join(HERE, "golden", "attention_mask_figure.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            a = line.split()
            if a[0] == "posid":
                pos = [int(x) for x in a[1:]]
            elif a[0] != "names":
                rows.append([c == "1" for c in a[1]])
    return np.array(rows), pos


def _two_blocks(dr, st, w, second_start_depth):
    """Block 1 from the root, then block 2 from the block-1 chain node at
    the given depth (1-based)."""
    tree = DraftTree(st.root, 1000)
    rows = []
    seg = dr.new_segment(w.K * 2)
    s1 = specdec.Start(0, st.root, st.T, dr.cond_from_taps(st.cond_taps), [])
    specdec.expand_block(dr, st, tree, rows, seg, [s1], w.K, 1,
                         (1, 1, 1, 1))
    node = [i for i, n in enumerate(tree.nodes)
            if n.depth == second_start_depth and n.rank == 1][0]
    s2 = specdec.start_from_node(tree, rows, st, node)
    rec = specdec.expand_block(dr, st, tree, rows, seg, [s2], w.K, 2,
                               (1, 1, 1, 1))
    return tree, rows, seg, s2, rec


def test_attention_pattern_matches_paper_figure():
    """The 8x8 block part of the App. A.2 figure (block rows against block
    columns) and the block rows' position ids.  The figure's two prefix
    columns (t1, t2) are deliberately left unpinned: the committed prefix
    is fully visible to every block row by construction, and position 0
    (t1) has no drafter K/V entry here, since no draft forward can have
    produced it (prefix entries come from each committed position's own
    draft forward, and position 0 precedes every draft)."""
    golden, pos = _read_golden()
    w = synth.Workload("fig", "f32", SHAPE, 1, K=4, M=2, B_max=1, budget=40,
                       n_seqs=1, prompt_len=(1, 1))
    _, _, tgt, dr = _models(w)
    # prompt of one token: the root t2 sits at position 1 as in the figure
    st = specdec.prefill(tgt, dr, [7])
    assert st.T == 1
    tree, rows, seg, s2, _ = _two_blocks(dr, st, w, 2)   # from B_{1,1}
    assert [r.pos for r in rows] == pos[2:]
    vis = np.zeros((8, 8), dtype=bool)
    for i, r in enumerate(rows):
        vis[i, r.vis] = True
    np.testing.assert_array_equal(vis, golden[2:, 2:])


def test_masked_rows_do_not_leak():
    """Numerically: off-path block-1 rows do not reach block 2; on-path rows
    and the prefix do."""
    _, _, tgt, dr = _models()
    st = specdec.prefill(tgt, dr, synth.prompts(W)[0])
    tree, rows, seg, s2, rec = _two_blocks(dr, st, W, 2)
    base = rec["logits"].copy()

    def rerun(mut):
        seg2 = dr.new_segment(8)
        for layer in range(1):
            seg2.k[layer][:4] = seg.k[layer][:4]
            seg2.v[layer][:4] = seg.v[layer][:4]
        mut(seg2)
        R = 4
        z, _ = dr.forward(s2.cond[None], [s2.token], np.zeros(R, int),
                          np.arange(1, 5), np.array([0, 0, 1, 2]),
                          [r.pos for r in rows[4:]], 4 + np.arange(R),
                          [r.vis for r in rows[4:]], st.dkv, seg2)
        return z

    same = rerun(lambda s: None)
    np.testing.assert_allclose(same, base, rtol=1e-12, atol=1e-12)

    def bump(i):
        def f(s):
            s.v[0][i] += 1.0
        return f
    for off_path in (2, 3):
        np.testing.assert_allclose(rerun(bump(off_path)), base, rtol=0,
                                   atol=0)
    for on_path in (0, 1):
        assert np.abs(rerun(bump(on_path)) - base).max() > 1e-6


def _hf_inputs(dr, conds, tokens, ks):
    """Shifted layer-0 inputs x = W_shift [h0_k, h0_{k-1}] (Eq. 2, Eq. 3)
    for rows given as (cond, token, k) with k-1 partner in the same list
    (or itself when k = 1), in torch ops."""
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))  # noqa
    eps = dr.shape.norm_eps
    d = dr.shape.d_model
    rms = lambda x, g: torch.nn.functional.rms_norm(x, (d,), t(g), eps)  # noqa
    h0 = []
    for c, y, k in zip(conds, tokens, ks):
        inp = torch.cat([rms(t(c), dr.norm_c), rms(t(dr.embed[y]), dr.norm_e),
                         rms(t(dr.pos_query[k - 1]), dr.norm_q)])
        h0.append(torch.nn.functional.linear(inp, t(dr.w_fuse)))
    xs = []
    for i, k in enumerate(ks):
        prev = h0[i - 1] if k > 1 else h0[i]
        xs.append(torch.nn.functional.linear(torch.cat([h0[i], prev]),
                                             t(dr.shift[0])))
    return torch.stack(xs)


@pytest.mark.parametrize("start_depth", [1, 2, 4])
def test_blocks_equal_causal_library_run_over_path(hf, start_depth):
    """Block 1 (after the catch-up prefix) and block 2 started from the
    chain node at ``start_depth`` equal a causal library Llama run over
    [catch-up inputs, block-1 rows up to the start, block-2 rows]."""
    tw, dw, tgt, dr = _models()
    prompt = synth.prompts(W)[0]
    st = specdec.prefill(tgt, dr, prompt)
    tree, rows, seg, s2, rec2 = _two_blocks(dr, st, W, start_depth)
    T = st.T
    # target taps from the library model, for the catch-up conditions
    tm = target_model(hf, SHAPE, tw)
    _, outs = layer_outputs(tm, input_ids=torch.tensor(prompt)[None])
    taps = [torch.stack([outs[li][0, j] for li in W.tap_layers]).numpy()
            for j in range(T)]
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))  # noqa
    conds = [np.zeros(SHAPE.d_model)] + [
        torch.nn.functional.linear(t(taps[p - 2].reshape(-1)),
                                   t(dr.w_cond)).numpy()
        for p in range(2, T + 1)]
    conds.append(torch.nn.functional.linear(t(taps[T - 1].reshape(-1)),
                                            t(dr.w_cond)).numpy())
    toks = list(prompt) + [st.root]
    x_pre = _hf_inputs(dr, conds[:T], toks[:T], [1] * T)
    x_b1 = _hf_inputs(dr, [conds[T]] * W.K, [st.root] * W.K,
                      list(range(1, W.K + 1)))
    m = drafter_trunk(hf, SHAPE, dw, 1, tw["embed"])
    seq = torch.cat([x_pre, x_b1])[None]
    pos = torch.arange(1, T + W.K + 1)[None]
    with torch.no_grad():
        ref1, outs1 = layer_outputs(m, inputs_embeds=seq, position_ids=pos)
    z1 = np.stack([rows[i].logits for i in range(W.K)])
    ref1 = ref1[0, T:].numpy()
    assert np.abs(z1 - ref1).max() <= 2e-6 * np.abs(ref1).max()
    # block 2: condition = the library's last-layer state at the start row
    h_start = outs1[-1][0, T + start_depth - 1].numpy()
    np.testing.assert_allclose(s2.cond, h_start, rtol=1e-5,
                               atol=1e-5 * np.abs(h_start).max())
    x_b2 = _hf_inputs(dr, [h_start] * W.K, [s2.token] * W.K,
                      list(range(1, W.K + 1)))
    seq2 = torch.cat([x_pre, x_b1[:start_depth], x_b2])[None]
    pos2 = torch.cat([torch.arange(1, T + start_depth + 1),
                      torch.arange(T + start_depth + 1,
                                   T + start_depth + W.K + 1)])[None]
    with torch.no_grad():
        ref2 = m(inputs_embeds=seq2, position_ids=pos2).logits[0, -W.K:]
    ref2 = ref2.numpy()
    assert np.abs(rec2["logits"] - ref2).max() <= 2e-6 * np.abs(ref2).max()


def _block(dr, K, cond, token, pos0, prefix, q=None):
    if q is not None:
        dr.pos_query = q
    R = K
    seg = dr.new_segment(R)
    idx = np.arange(R)
    return dr.forward(cond[None], [token], np.zeros(R, int), idx + 1,
                      np.where(idx > 0, idx - 1, idx), pos0 + 1 + idx, idx,
                      [list(range(r + 1)) for r in idx], prefix, seg)


def test_prefix_consistency_and_causality_in_k():
    _, _, tgt, dr = _models()
    st = specdec.prefill(tgt, dr, synth.prompts(W)[0])
    c = dr.cond_from_taps(st.cond_taps)
    z4, h4 = _block(dr, 4, c, st.root, st.T, st.dkv)
    for kp in (1, 2, 3):
        zk, hk = _block(dr, kp, c, st.root, st.T, st.dkv)
        np.testing.assert_allclose(zk, z4[:kp], rtol=1e-12, atol=1e-12)
    q = dr.pos_query.copy()
    q2 = q.copy()
    q2[3] += 0.5
    z4b, _ = _block(dr, 4, c, st.root, st.T, st.dkv, q2)
    dr.pos_query = q
    np.testing.assert_allclose(z4b[:3], z4[:3], rtol=1e-12, atol=1e-12)
    assert np.abs(z4b[3] - z4[3]).max() > 1e-6


def test_start_permutation_invariance():
    _, _, tgt, dr = _models()
    st = specdec.prefill(tgt, dr, synth.prompts(W)[0])
    rng = np.random.default_rng(3)
    B, K = 3, W.K
    conds = rng.standard_normal((B, SHAPE.d_model))
    toks = rng.integers(0, SHAPE.vocab, B)

    def run(order):
        R = B * K
        rs = np.repeat(np.arange(B), K)
        rk = np.tile(np.arange(1, K + 1), B)
        idx = np.arange(R)
        seg = dr.new_segment(R)
        vis = [[s * K + j for j in range(k)] for s, k in zip(rs, rk)]
        return dr.forward(conds[order], toks[order], rs, rk,
                          np.where(rk > 1, idx - 1, idx),
                          st.T + rk, idx, vis, st.dkv, seg)[0]
    a = run(np.arange(B))
    perm = np.array([2, 0, 1])
    b = run(perm)
    for i, s in enumerate(perm):
        np.testing.assert_allclose(b[i * K:(i + 1) * K], a[s * K:(s + 1) * K],
                                   rtol=1e-12, atol=1e-12)


def test_later_blocks_bypass_w_cond():
    _, _, tgt, dr = _models()
    st = specdec.prefill(tgt, dr, synth.prompts(W)[0])
    tree, rows, seg, s2, rec = _two_blocks(dr, st, W, 3)
    node = tree.nodes[s2.node]
    assert s2.cond is rows[node.row].h_last
    dr.w_cond = np.full_like(dr.w_cond, np.nan)
    z, _ = dr.forward(s2.cond[None], [s2.token], np.zeros(4, int),
                      np.arange(1, 5), np.array([0, 0, 1, 2]),
                      [r.pos for r in rows[4:]], 4 + np.arange(4),
                      [r.vis for r in rows[4:]], st.dkv, seg)
    assert np.isfinite(z).all()
    np.testing.assert_allclose(z, rec["logits"], rtol=1e-12, atol=1e-12)
