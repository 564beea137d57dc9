"""Draft tree, rank-guided sibling attachment and next-block starts (oracle).

Test infrastructure: see the package docstring.

Readings taken here (the paper describes these steps in prose only,
Sec. 3.2 and Alg. 2):
* Within a block, the rank-1 token of row k is the *chain* node and its
  ranks 2..b are siblings under the same parent; the parent of row k's
  tokens is the chain node of row k-1 (the start node for k = 1).  A row
  with b = 0 ends its block's chain: later rows of that block attach nothing.
* The tree budget counts the root.  Nodes are inserted in the order
  (block, k, start, rank) until the budget is reached; there is no pruning.
* Next-block starts: first the chain end (k = K) of each block in start
  order, then sibling nodes (rank >= 2) of rows whose bucket is b1 or b2, by
  cumulative log-probability (descending, ties to the lower node index);
  at most B_max, none once the tree is full.  (Parity unpinned: the paper
  does not give the rule.)
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass
class Node:
    token: int
    parent: int          # -1 for the root
    depth: int
    row: int             # drafter row that proposed it; -1 for the root
    rank: int            # 1-based rank in that row's distribution; 0: root
    logp: float
    cum_logp: float


class DraftTree:
    def __init__(self, root_token: int, budget: int):
        self.budget = budget
        self.nodes = [Node(int(root_token), -1, 0, -1, 0, 0.0, 0.0)]

    def __len__(self):
        return len(self.nodes)

    def full(self) -> bool:
        return len(self.nodes) >= self.budget

    def add(self, token, parent, row, rank, logp) -> int:
        p = self.nodes[parent]
        self.nodes.append(Node(int(token), parent, p.depth + 1, row, rank,
                               float(logp), p.cum_logp + float(logp)))
        return len(self.nodes) - 1

    def anc_or_self(self, i: int) -> list:
        out = []
        while i >= 0:
            out.append(i)
            i = self.nodes[i].parent
        return out[::-1]

    def children(self, i: int) -> list:
        return [j for j, n in enumerate(self.nodes) if n.parent == i]

    def mask(self) -> np.ndarray:
        """[n, n] bool: mask[i, j] iff node j is an ancestor-or-self of i."""
        n = len(self.nodes)
        m = np.zeros((n, n), dtype=bool)
        for i in range(n):
            m[i, self.anc_or_self(i)] = True
        return m


@dataclasses.dataclass
class Start:
    """One next-block starting point (a tree node) and what it carries."""
    node: int
    token: int
    pos: int                 # RoPE position of the start node
    cond: np.ndarray         # [d] condition vector before norm_c
    anc_rows: list           # iteration rows visible to the new block


@dataclasses.dataclass
class DraftRow:
    """One drafter row of the current iteration (block position k of a start)."""
    block: int
    start: int               # index of its start within its block
    start_node: int
    k: int                   # 1-based block position
    pos: int                 # RoPE position = start pos + k
    vis: list                # iteration rows it attends to (incl. itself)
    logits: np.ndarray = None
    h_last: np.ndarray = None
    lse: float = 0.0
    topk: np.ndarray = None      # top-10 target token ids
    topk_d: np.ndarray = None    # the same as drafter output ids
    psi: np.ndarray = None
    scores: np.ndarray = None
    bucket: int = -1
    branch: int = 0


def attach_block(tree: DraftTree, rows: list, block_rows: list, n_starts,
                 start_nodes, K: int):
    """Attach the top-b tokens of every row of one block (Alg. 2, inner
    loop), in (k, start, rank) order within the budget.

    block_rows[s][k-1] is the row id of start s at position k.
    Returns (alive, chain): whether start s's chain reached k = K, and the
    last chain node of each start.
    """
    alive = [True] * n_starts
    chain = list(start_nodes)
    for k in range(1, K + 1):
        for s in range(n_starts):
            if not alive[s]:
                continue
            r = rows[block_rows[s][k - 1]]
            parent = chain[s]
            got_chain = False
            for rank in range(1, r.branch + 1):
                if tree.full():
                    break
                tok = int(r.topk[rank - 1])
                n = tree.add(tok, parent, block_rows[s][k - 1], rank,
                             r.logits[r.topk_d[rank - 1]] - r.lse)
                if rank == 1:
                    chain[s] = n
                    got_chain = True
            if not got_chain:
                alive[s] = False
    return alive, chain


def select_starts(tree: DraftTree, rows: list, alive, chain, first_new: int,
                  B_max: int) -> list:
    """Nodes that start the next block (see the module docstring)."""
    if tree.full():
        return []
    ends = [chain[s] for s in range(len(alive)) if alive[s]]
    sib = [n for n in range(first_new, len(tree.nodes))
           if tree.nodes[n].rank >= 2 and rows[tree.nodes[n].row].bucket
           in (1, 2)]
    sib.sort(key=lambda n: (-tree.nodes[n].cum_logp, n))
    return (ends + sib)[:B_max]


def accept(tree: DraftTree, greedy) -> tuple:
    """Greedy acceptance walk (Alg. 2, verify line): from the root, follow
    the child whose token equals the target's greedy choice at the current
    node; the target's choice at the last accepted node is the bonus token.

    Returns (path of accepted node ids, bonus token).  Children of one node
    carry distinct tokens by construction; if they did not, the lowest node
    index would win.
    """
    cur, path = 0, []
    while True:
        nxt = [c for c in tree.children(cur)
               if tree.nodes[c].token == int(greedy[cur])]
        if not nxt:
            break
        cur = min(nxt)
        path.append(cur)
    return path, int(greedy[cur])
