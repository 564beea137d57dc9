"""Pins of the oracle's target forward and tree verification.

* causal prefill == transformers' Llama (library implementation of the
  decoder the paper's target follows), logits and per-layer taps;
* a single-chain tree reproduces causal attention exactly (its rows equal the
  causal rows of the same tokens);
* every tree node's verify logits equal a causal forward over
  prefix + root-to-node path (brute force over paths on a small tree).
"""
import numpy as np
import pytest
import torch

import synth
from oracle.model import Target
from oracle.tree import DraftTree

from hfref import layer_outputs, target_model

SHAPE_GQA = synth.ModelShape(3, 64, 4, 2, 16, 96, 211)


def _target(shape, dtype="f32", seed=0):
    tw = synth.make_weights(synth.target_specs(shape), seed, dtype,
                            jitter=0.1)
    taps = (0, shape.n_layers // 2, shape.n_layers - 1)
    return tw, Target(tw, shape, dtype, taps)


def _causal(target, tokens):
    n = len(tokens)
    idx = np.arange(n)
    seg = target.new_segment(n)
    return target.forward(tokens, idx, idx, [list(range(r + 1)) for r in idx],
                          target.new_prefix(), seg), seg


@pytest.mark.parametrize("shape", [SHAPE_GQA, synth.TINY])
def test_causal_forward_matches_transformers(hf, shape):
    tw, tgt = _target(shape)
    toks = np.random.default_rng(5).integers(0, shape.vocab, 19)
    (logits, taps), _ = _causal(tgt, toks)
    m = target_model(hf, shape, tw)
    ref, outs = layer_outputs(m, input_ids=torch.tensor(toks)[None])
    ref = ref[0].numpy()
    scale = np.abs(ref).max()
    # transformers computes RMSNorm statistics and RoPE tables in float32
    assert np.abs(logits - ref).max() <= 2e-6 * scale
    for j, layer in enumerate(tgt.tap_layers):
        t = outs[layer][0].numpy()
        assert np.abs(taps[:, j] - t).max() <= 2e-6 * np.abs(t).max()


def test_prefix_plus_rows_equals_causal():
    """Rows run on top of a committed prefix give the causal results."""
    _, tgt = _target(SHAPE_GQA)
    toks = np.random.default_rng(6).integers(0, SHAPE_GQA.vocab, 12)
    (full, _), seg = _causal(tgt, toks)
    pre = tgt.new_prefix()
    for layer in range(SHAPE_GQA.n_layers):
        for i in range(7):
            pre.append(layer, seg.k[layer][i], seg.v[layer][i])
    rest = np.arange(7, 12)
    s2 = tgt.new_segment(5)
    lg, _ = tgt.forward(toks[7:], rest, np.arange(5),
                        [list(range(r + 1)) for r in range(5)], pre, s2)
    np.testing.assert_allclose(lg, full[7:], rtol=1e-10, atol=1e-10)


def _random_tree(rng, root, budget, vocab):
    tree = DraftTree(root, budget)
    while not tree.full():
        parent = int(rng.integers(0, len(tree)))
        tree.add(int(rng.integers(0, vocab)), parent, -1, 1, 0.0)
    return tree


def _verify(tgt, prefix_toks, tree):
    (_, _), seg = _causal(tgt, prefix_toks)
    pre = tgt.new_prefix()
    T = len(prefix_toks)
    for layer in range(tgt.shape.n_layers):
        for i in range(T):
            pre.append(layer, seg.k[layer][i], seg.v[layer][i])
    n = len(tree)
    s = tgt.new_segment(n)
    pos = np.array([T + nd.depth for nd in tree.nodes])
    return tgt.forward([nd.token for nd in tree.nodes], pos, np.arange(n),
                       [tree.anc_or_self(i) for i in range(n)], pre, s)


def test_single_chain_tree_is_causal():
    """A tree that is a single chain is plain causal attention."""
    _, tgt = _target(SHAPE_GQA)
    rng = np.random.default_rng(7)
    toks = rng.integers(0, SHAPE_GQA.vocab, 15)
    tree = DraftTree(int(toks[9]), 6)
    for j in range(5):
        tree.add(int(toks[10 + j]), j, -1, 1, 0.0)
    lg, taps = _verify(tgt, toks[:9], tree)
    (full, ftaps), _ = _causal(tgt, toks)
    np.testing.assert_allclose(lg, full[9:], rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(taps, ftaps[9:], rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tree_verify_equals_path_bruteforce(hf, seed):
    """Tree verification: each node's logits equal a causal forward of
    the library model over prefix + the root-to-node path."""
    tw, tgt = _target(SHAPE_GQA, seed=seed)
    rng = np.random.default_rng(10 + seed)
    prefix = rng.integers(0, SHAPE_GQA.vocab, 8)
    tree = _random_tree(rng, int(rng.integers(0, SHAPE_GQA.vocab)), 14,
                        SHAPE_GQA.vocab)
    lg, _ = _verify(tgt, prefix, tree)
    m = target_model(hf, SHAPE_GQA, tw)
    for i in range(len(tree)):
        path = [tree.nodes[j].token for j in tree.anc_or_self(i)]
        seq = np.concatenate([prefix, path])
        with torch.no_grad():
            ref = m(input_ids=torch.tensor(seq)[None]).logits[0, -1].numpy()
        assert np.abs(lg[i] - ref).max() <= 2e-6 * np.abs(ref).max()


def test_bf16_numerics_stay_close_to_f64():
    """The bf16 rounding model perturbs logits by well under the 2e-2
    relative bound the bf16 configurations are held to."""
    tw32, t64 = _target(SHAPE_GQA, "bf16")
    t_b = Target(tw32, SHAPE_GQA, "bf16", t64.tap_layers)
    t_f = Target(tw32, SHAPE_GQA, "f32", t64.tap_layers)
    toks = np.random.default_rng(8).integers(0, SHAPE_GQA.vocab, 10)
    (lb, _), _ = _causal(t_b, toks)
    (lf, _), _ = _causal(t_f, toks)
    rel = np.abs(lb - lf).max(axis=1) / np.abs(lf).max(axis=1)
    assert rel.max() < 2e-2
    assert rel.max() > 0       # the rounding is actually applied
