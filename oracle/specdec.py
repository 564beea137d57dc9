"""Prefill, one SpecBlock verifier iteration, and plain greedy decoding
(oracle).

Test infrastructure: see the package docstring.

Positions and caches (our reading of the attention-mask figure of App. A.2):
* the target's prefix holds K/V for positions 0..T-1; the root x_T (the
  last verified token, not yet run through the target) sits at position T;
* drafter row k of a block started at node n sits at RoPE position
  pos(n) + k and predicts the token at that position;
* the drafter's prefix holds one entry per position 1..T: the K/V of the
  drafter row at that position along the committed path.  An accepted draft
  node reuses the K/V of the row that proposed it (its own draft forward);
  the bonus position reuses the row that continued the last accepted node,
  when the tree has one.  Positions no draft forward covered (the prompt,
  and a bonus with no continuing row) get a *catch-up* row: a K = 1 block
  started at the previous position, conditioned on the target taps of the
  position before that (zero for position 1), attending causally;
* block 1 of an iteration starts at the root with c = W_cond [taps at T-1]
  (Eq. 1); later blocks start at tree nodes with the cached h^(L) of the row
  that proposed the node and bypass W_cond (Sec. 3.2);
* tree nodes are verified at position T + depth, each attending to the
  target prefix and its ancestors-or-self; the root and accepted nodes keep
  the K/V computed during verification.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .model import Drafter, Prefix, Target
from .rank import TOPK, bucket_of_scores, psi, rank_scores, topk_ids
from .numerics import logsumexp
from .sampling import accept_sample
from .tree import (DraftRow, DraftTree, Start, accept, attach_block,
                   select_starts)


def argmax_low(z) -> int:
    """argmax with ties to the smallest id."""
    return int(np.argmax(np.asarray(z)))


@dataclasses.dataclass
class SeqState:
    tokens: list             # committed stream, prompt included, root last
    T: int                   # root position == #target prefix entries
    root: int
    tkv: Prefix              # target K/V, positions 0..T-1
    dkv: Prefix              # drafter K/V, positions 1..T
    cond_taps: np.ndarray    # [3, d] target taps at position T-1


def _copy_in(prefix: Prefix, seg, idx):
    for layer in range(len(prefix.k)):
        for i in idx:
            prefix.append(layer, seg.k[layer][i], seg.v[layer][i])


def catch_up(drafter: Drafter, conds, tokens, pos0: int, prefix: Prefix):
    """Catch-up rows for consecutive positions pos0+1, pos0+2, ...: row j is a
    K = 1 block started at position pos0+j with condition conds[j] and token
    tokens[j]; rows attend to ``prefix`` and causally to each other.
    Returns the filled drafter segment."""
    n = len(tokens)
    seg = drafter.new_segment(n)
    idx = np.arange(n)
    drafter.forward(conds, tokens, idx, np.ones(n, np.int64), idx,
                    pos0 + 1 + idx, idx, [list(range(r + 1)) for r in idx],
                    prefix, seg)
    return seg


def prefill(target: Target, drafter: Drafter, prompt) -> SeqState:
    """Causal target forward over the prompt x_0..x_{T0-1}; the root x_{T0}
    is its greedy token; drafter entries 1..T0 are catch-up rows."""
    prompt = [int(t) for t in prompt]
    T0 = len(prompt)
    seg = target.new_segment(T0)
    idx = np.arange(T0)
    logits, taps = target.forward(prompt, idx, idx,
                                  [list(range(r + 1)) for r in idx],
                                  target.new_prefix(), seg)
    tkv = target.new_prefix()
    _copy_in(tkv, seg, idx)
    root = argmax_low(logits[-1])
    d = target.shape.d_model
    conds = np.zeros((T0, d))
    for p in range(2, T0 + 1):
        conds[p - 1] = drafter.cond_from_taps(taps[p - 2])
    dseg = catch_up(drafter, conds, prompt, 0, drafter.new_prefix())
    dkv = drafter.new_prefix()
    _copy_in(dkv, dseg, idx)
    return SeqState(prompt + [root], T0, root, tkv, dkv, taps[T0 - 1])


def expand_block(drafter: Drafter, st: SeqState, tree: DraftTree, rows: list,
                 seg, starts: list, K: int, block: int, branch_map,
                 forced=None):
    """One block expansion (one batched drafter forward over all starts),
    followed by psi, the rank head, branching and sibling attachment.
    ``forced``, when given, replaces the rank head's bucket of row r (row id
    within this iteration) by forced[r] clamped to 0..3; the scores are still
    computed.  Returns a record of everything the step computed."""
    base = len(rows)
    block_rows = []
    for s, sp in enumerate(starts):
        ids = []
        for k in range(1, K + 1):
            rid = base + s * K + (k - 1)
            vis = list(sp.anc_rows) + [base + s * K + j for j in range(k)]
            rows.append(DraftRow(block, s, sp.node, k, sp.pos + k, vis))
            ids.append(rid)
        block_rows.append(ids)
    new = rows[base:]
    R = len(new)
    local = np.arange(R)
    row_start = np.array([r.start for r in new])
    row_k = np.array([r.k for r in new])
    row_pred = np.where(row_k > 1, local - 1, local)
    z, h = drafter.forward(np.stack([sp.cond for sp in starts]),
                           [sp.token for sp in starts], row_start, row_k,
                           row_pred, np.array([r.pos for r in new]),
                           base + local, [r.vis for r in new], st.dkv, seg)
    for i, r in enumerate(new):
        r.logits, r.h_last = z[i], h[i]
        r.lse = float(logsumexp(z[i]))
        r.topk_d = topk_ids(z[i], TOPK)
        r.topk = drafter.to_target(r.topk_d)
        r.psi = psi(z[i])
        r.scores = rank_scores(drafter.rank_w, drafter.rank_b, h[i], r.psi)
        r.bucket = (bucket_of_scores(r.scores) if forced is None
                    else min(max(int(forced[base + i]), 0), 3))
        r.branch = int(branch_map[r.bucket])
    first_new = len(tree.nodes)
    alive, chain = attach_block(tree, rows, block_rows, len(starts),
                                [sp.node for sp in starts], K)
    return dict(block=block, base=base, R=R, block_rows=block_rows,
                alive=alive, chain=chain, first_new=first_new,
                logits=z, h_last=h)


def start_from_node(tree: DraftTree, rows: list, st: SeqState, n: int):
    """A later-block start at node n: cached h^(L) of the row that proposed
    it (no W_cond), the node's own token, and that row's visible rows."""
    node = tree.nodes[n]
    r = rows[node.row]
    return Start(n, node.token, st.T + node.depth, r.h_last, list(r.vis))


def continuing_row(tree: DraftTree, rows: list, n: int, K: int):
    """Row at position pos(n) + 1 on a path through node n, if any: the next
    row of n's block when n is a chain node short of K, else row 1 of a block
    started at n."""
    if n > 0:
        node = tree.nodes[n]
        r = rows[node.row]
        if node.rank == 1 and r.k < K:
            for j, q in enumerate(rows):
                if q.block == r.block and q.start == r.start and \
                        q.k == r.k + 1:
                    return j
    for j, q in enumerate(rows):
        if q.start_node == n and q.k == 1:
            return j
    return None


def reject_signal(drafter: Drafter, tree: DraftTree, rows: list, path: list,
                  bonus: int, K: int):
    """The verifier-derived signal's r at the rejected position (Sec. 3.4,
    Eq. 8): the drafter's probability of the target's token (the bonus) at
    the position after the last accepted node, from the drafter row that
    predicted that position (the row continuing that node).  None when no
    row did; 0 when the bonus is outside a reduced drafter vocabulary."""
    cur = path[-1] if path else 0
    j = continuing_row(tree, rows, cur, K)
    if j is None:
        return None
    z = rows[j].logits
    if drafter.d2t is None:
        idx = bonus
    else:
        idx = int(np.searchsorted(drafter.d2t, bonus))
        if idx >= len(drafter.d2t) or drafter.d2t[idx] != bonus:
            return 0.0
    return float(np.exp(z[idx] - logsumexp(z)))


def iteration(target: Target, drafter: Drafter, st: SeqState, w,
              branch_map=None, plant=None, buckets=None,
              sampling=None) -> dict:
    """One verifier iteration (Alg. 2) for one sequence; mutates ``st``.

    ``plant(tree, rows)``, when given, may rewrite node tokens after drafting
    and before verification (tests plant known continuations with it).
    ``buckets``, when given, forces the bucket of every drafter row of this
    iteration (indexed by row id), a synthetic workload knob.
    ``sampling`` = (temperature, u_acc, u_bonus) replaces greedy acceptance
    by stochastic tree verification (``sampling.accept_sample``)."""
    branch_map = tuple(branch_map or w.branch_map)
    K = w.K
    tree = DraftTree(st.root, w.budget)
    rows: list = []
    seg = drafter.new_segment(w.rows_per_seq)
    starts = [Start(0, st.root, st.T, drafter.cond_from_taps(st.cond_taps),
                    [])]
    expansions = []
    for m in range(1, w.M + 1):
        if not starts:
            break
        rec = expand_block(drafter, st, tree, rows, seg, starts, K, m,
                           branch_map, buckets)
        rec["starts"] = starts
        expansions.append(rec)
        if m < w.M:
            picks = select_starts(tree, rows, rec["alive"], rec["chain"],
                                  rec["first_new"], w.B_max)
            starts = [start_from_node(tree, rows, st, n) for n in picks]
        else:
            starts = []
    if plant is not None:
        plant(tree, rows)
    # tree verification: one target forward over all nodes
    n = len(tree.nodes)
    tseg = target.new_segment(n)
    pos = np.array([st.T + nd.depth for nd in tree.nodes])
    vlogits, vtaps = target.forward([nd.token for nd in tree.nodes], pos,
                                    np.arange(n),
                                    [tree.anc_or_self(i) for i in range(n)],
                                    st.tkv, tseg)
    greedy = np.array([argmax_low(z) for z in vlogits])
    if sampling is None:
        path, bonus = accept(tree, greedy)
    else:
        smp = accept_sample(tree, vlogits, *sampling)
        path, bonus = smp["path"], smp["bonus"]
    r_reject = reject_signal(drafter, tree, rows, path, bonus, K)
    # commit
    T = st.T
    keep = [0] + path
    _copy_in(st.tkv, tseg, keep)
    _copy_in(st.dkv, seg, [tree.nodes[p].row for p in path])
    cur = keep[-1]
    cont = continuing_row(tree, rows, cur, K)
    fallback = cont is None
    if fallback:
        parent = tree.nodes[cur].parent
        cond = drafter.cond_from_taps(vtaps[parent])
        fseg = catch_up(drafter, cond[None], [tree.nodes[cur].token],
                        T + len(path), st.dkv)
        _copy_in(st.dkv, fseg, [0])
    else:
        _copy_in(st.dkv, seg, [cont])
    committed = [tree.nodes[p].token for p in path] + [bonus]
    st.tokens += committed
    st.T = T + len(path) + 1
    st.root = bonus
    st.cond_taps = vtaps[cur]
    return dict(tree=tree, rows=rows, expansions=expansions,
                verify_logits=vlogits, greedy=greedy, taps=vtaps, path=path,
                bonus=bonus, tau=len(path) + 1, committed=committed,
                r_reject=r_reject,
                fallback=fallback, T_before=T)


def speculative_decode(target: Target, drafter: Drafter, prompt, w,
                       n_new: int, branch_map=None, plant=None, buckets=None,
                       sampling=None):
    """Prefill, then iterate until at least n_new tokens are committed.
    ``buckets(i)``, when given, returns the forced buckets of iteration i;
    ``sampling(i)`` the (temperature, u_acc, u_bonus) of iteration i."""
    st = prefill(target, drafter, prompt)
    out = [st.root]
    taus = []
    while len(out) < n_new:
        i = len(taus)
        rec = iteration(target, drafter, st, w, branch_map, plant,
                        None if buckets is None else buckets(i),
                        None if sampling is None else sampling(i))
        out += rec["committed"]
        taus.append(rec["tau"])
    return out[:n_new], taus


def greedy_decode(target: Target, prompt, n_new: int) -> list:
    """The target's own greedy continuation, one position per forward with a
    K/V cache (the lossless reference)."""
    prompt = [int(t) for t in prompt]
    T0 = len(prompt)
    seg = target.new_segment(T0)
    idx = np.arange(T0)
    logits, _ = target.forward(prompt, idx, idx,
                               [list(range(r + 1)) for r in idx],
                               target.new_prefix(), seg)
    kv = target.new_prefix()
    _copy_in(kv, seg, idx)
    out = [argmax_low(logits[-1])]
    while len(out) < n_new:
        s1 = target.new_segment(1)
        lg, _ = target.forward([out[-1]], [len(kv)], [0], [[0]], kv, s1)
        _copy_in(kv, s1, [0])
        out.append(argmax_low(lg[0]))
    return out
