"""Property pins of the tree builder and the acceptance walk."""
import numpy as np
from hypothesis import given, settings, strategies as st

from oracle.tree import (DraftRow, DraftTree, accept, attach_block,
                         select_starts)


def _rows(draw_branch, draw_bucket, rng, n_starts, K, vocab):
    rows, block_rows = [], []
    for s in range(n_starts):
        ids = []
        for k in range(1, K + 1):
            r = DraftRow(1, s, 0, k, k, [])
            z = rng.standard_normal(vocab)
            r.logits = z
            r.lse = float(np.log(np.exp(z).sum()))
            r.topk = np.argsort(-z, kind="stable")[:10]
            r.topk_d = r.topk
            r.bucket = draw_bucket()
            r.branch = draw_branch(r.bucket)
            ids.append(len(rows))
            rows.append(r)
        block_rows.append(ids)
    return rows, block_rows


@settings(max_examples=200, deadline=None)
@given(seed=st.integers(0, 10 ** 6), n_starts=st.integers(1, 6),
       K=st.integers(1, 6), budget=st.integers(1, 60),
       bmap=st.sampled_from([(2, 4, 10, 0), (2, 4, 6, 4), (1, 1, 1, 1)]),
       B_max=st.integers(1, 8))
def test_attach_and_select_invariants(seed, n_starts, K, budget, bmap, B_max):
    rng = np.random.default_rng(seed)
    rows, block_rows = _rows(lambda b: bmap[b],
                             lambda: int(rng.integers(0, 4)), rng, n_starts,
                             K, 50)
    tree = DraftTree(0, budget)
    # start nodes: the root for start 0, otherwise fresh depth-1 nodes
    starts = [0]
    for s in range(1, n_starts):
        if not tree.full():
            starts.append(tree.add(1000 + s, 0, -1, 2, -1.0))
    n_starts = len(starts)
    first_new = len(tree)
    alive, chain = attach_block(tree, rows, block_rows[:n_starts], n_starts,
                                starts, K)
    nodes = tree.nodes
    assert len(tree) <= budget
    order = []
    for i in range(first_new, len(tree)):
        nd = nodes[i]
        assert 0 <= nd.parent < i
        assert nd.depth == nodes[nd.parent].depth + 1
        r = rows[nd.row]
        s = r.start
        assert nd.depth == nodes[starts[s]].depth + r.k
        assert 1 <= nd.rank <= r.branch
        assert nd.token == r.topk[nd.rank - 1]
        assert np.isclose(nd.cum_logp, nodes[nd.parent].cum_logp + nd.logp)
        # the parent is the start (k = 1) or the rank-1 node of row k-1
        if r.k == 1:
            assert nd.parent == starts[s]
        else:
            p = nodes[nd.parent]
            assert p.rank == 1 and rows[p.row].k == r.k - 1 and \
                rows[p.row].start == s
        order.append((r.k, s, nd.rank))
    assert order == sorted(order)                   # (k, start, rank) order
    # a chain is alive iff its k = K rank-1 node exists
    for s in range(n_starts):
        if alive[s]:
            assert nodes[chain[s]].rank == 1 and rows[nodes[chain[s]].row].k \
                == K
    # rows whose chain survived attach min(b, room) tokens; if anything was
    # cut, the tree is full
    wanted = 0
    for s in range(n_starts):
        for k in range(1, K + 1):
            r = rows[block_rows[s][k - 1]]
            wanted += r.branch
            if r.branch == 0:
                break
    if len(tree) - first_new < wanted:
        assert tree.full() or any(not a for a in alive)
    picks = select_starts(tree, rows, alive, chain, first_new, B_max)
    assert len(picks) <= B_max
    if tree.full():
        assert picks == []
        return
    ends = [chain[s] for s in range(n_starts) if alive[s]]
    assert picks[:len(ends)] == ends[:B_max]
    sib = picks[len(ends):]
    for n in sib:
        assert nodes[n].rank >= 2 and rows[nodes[n].row].bucket in (1, 2)
    cl = [nodes[n].cum_logp for n in sib]
    assert cl == sorted(cl, reverse=True)


def _random_tree(rng, budget, vocab):
    tree = DraftTree(int(rng.integers(vocab)), budget)
    while not tree.full():
        p = int(rng.integers(len(tree)))
        used = {tree.nodes[c].token for c in tree.children(p)}
        free = [t for t in range(vocab) if t not in used]
        if not free:
            continue
        tree.add(int(rng.choice(free)), p, -1, 1, 0.0)
    return tree


@settings(max_examples=300, deadline=None)
@given(seed=st.integers(0, 10 ** 6), budget=st.integers(1, 40),
       vocab=st.integers(2, 6))
def test_accept_equals_bruteforce_over_paths(seed, budget, vocab):
    """Greedy acceptance (Alg. 2): the walk returns the longest root path whose
    every token is the target's greedy choice at its parent."""
    rng = np.random.default_rng(seed)
    tree = _random_tree(rng, budget, vocab)
    g = rng.integers(0, vocab, len(tree))
    path, bonus = accept(tree, g)
    best = []
    for leaf in range(len(tree)):
        anc = tree.anc_or_self(leaf)[1:]
        ok = []
        for n in anc:
            if tree.nodes[n].token != g[tree.nodes[n].parent]:
                break
            ok.append(n)
        if len(ok) > len(best):
            best = ok
    assert path == best
    last = path[-1] if path else 0
    assert bonus == g[last]
