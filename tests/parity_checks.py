"""Call-by-call comparison of one SpecBlock iteration on the device with the
oracle, for the bf16 configurations.

Every call runs on the oracle's inputs: before each call the device's tree
state (nodes, next-block starts, cached h^(L), greedy choices) is reset to the
oracle's (teacher forcing, oracle -> device only), so one near-tie cannot
change what later calls are given and every call of every sampled sequence is
compared.

The bar for one call:
* continuous outputs (logits, h^(L), taps, caches) within ``tol`` relative;
* discrete outputs are *valid* under the oracle's values up to the observed
  error E of that row: the device's i-th top-k id carries an oracle logit
  within 2E of the oracle's i-th largest (a perturbation of at most E per
  logit cannot do more), an argmax within 2E of the oracle's maximum, a
  bucket whose oracle score is within 2 x (score error) of the best;
* the device's own discrete outputs are exactly consistent with its own
  continuous outputs (top-k of its logits, ties to the smaller id; the
  branch of its bucket);
* where no bucket of a call met a near-tie, the tree the call built has
  the oracle's shape exactly, its tokens are the oracle's wherever the top-k
  ids agree, and the starts it picked are the oracle's up to near-ties of
  cumulative log-probability.
"""
from __future__ import annotations

import copy
import dataclasses

import numpy as np
import torch

from oracle import specdec

from gpu_harness import host, rel_err


@dataclasses.dataclass
class Tally:
    rows: int = 0
    rows_exact: int = 0
    calls_exact: int = 0
    calls_excused: int = 0
    worst_logit: float = 0.0
    worst_verify: float = 0.0

    def __str__(self):
        return (f"{self.rows_exact}/{self.rows} rows with identical top-b "
                f"and bucket; tree shape compared exactly in "
                f"{self.calls_exact} calls, {self.calls_excused} calls with a "
                f"bucket near-tie; worst "
                f"rel err draft logits {self.worst_logit:.2e}, verify "
                f"{self.worst_verify:.2e}")


def continuation(tgt, st, n):
    """The target's greedy tokens after the root of ``st`` (oracle forwards
    one position at a time on a copy of the prefix)."""
    kv = copy.deepcopy(st.tkv)
    tok, out = st.root, []
    for j in range(n):
        seg = tgt.new_segment(1)
        lg, _ = tgt.forward([tok], [st.T + j], [0], [[0]], kv, seg)
        for layer in range(len(kv.k)):
            kv.append(layer, seg.k[layer][0], seg.v[layer][0])
        tok = specdec.argmax_low(lg[0])
        out.append(tok)
    return out


def planter(stream, depth, vocab, snap):
    """plant() for specdec.iteration: keeps a copy of the drafted tree in
    ``snap``, then rewrites the lowest-id path of the given depth (or the
    deepest available) with the greedy continuation ``stream``; a tree of
    the root alone has no path to plant."""
    def plant(tree, rows):
        snap.append(copy.deepcopy(tree))
        if not depth:
            return
        dmax = max(nd.depth for nd in tree.nodes)
        want = min(depth, dmax)
        if want == 0:
            return
        leaf = min(i for i in range(1, len(tree)) if tree.nodes[i].depth == want)
        for j, nid in enumerate(tree.anc_or_self(leaf)[1:]):
            tok = stream[j]
            for c in tree.children(tree.nodes[nid].parent):
                if c != nid and tree.nodes[c].token == tok:
                    tree.nodes[c].token = (tok + 1) % vocab
            tree.nodes[nid].token = tok
    return plant


def oracle_iteration(tgt, dr, st, w, plant_depth=0, buckets=None):
    """One oracle iteration on a copy of ``st`` (``buckets``: forced row
    buckets); returns (state after, record, drafted tree before planting)."""
    after = copy.deepcopy(st)
    snap = []
    stream = continuation(tgt, st, plant_depth) if plant_depth else []
    rec = specdec.iteration(tgt, dr, after, w,
                            plant=planter(stream, plant_depth,
                                          w.target.vocab, snap),
                            buckets=buckets)
    return after, rec, snap[0]


def _anc_words(tree, n, bw):
    anc = np.zeros((n, bw), np.uint32)
    for i in range(n):
        for j in tree.anc_or_self(i):
            anc[i, j >> 5] |= np.uint32(1 << (j & 31))
    return anc


def inject_tree(rt, seq, tree, n, starts=None, rows=None):
    """Overwrite the device tree of ``seq`` with the oracle's first n nodes;
    given, also the next block's starts and the rows' cached h^(L)."""
    t = rt.tree
    nodes = tree.nodes[:n]
    col = lambda f, dt: torch.as_tensor(np.array([getattr(x, f) for x in nodes], dt))  # noqa: E731
    t["token"][seq, :n] = col("token", np.int32)
    t["parent"][seq, :n] = col("parent", np.int32)
    t["depth"][seq, :n] = col("depth", np.int32)
    t["row"][seq, :n] = col("row", np.int32)
    t["rank"][seq, :n] = col("rank", np.int32)
    t["logp"][seq, :n] = col("logp", np.float32)
    t["cum_logp"][seq, :n] = col("cum_logp", np.float32)
    bw = t["anc"].shape[-1]
    t["anc"][seq, :n] = torch.as_tensor(_anc_words(tree, n, bw).view(np.int32))
    t["n_nodes"][seq] = n
    if starts is not None:
        t["starts"][seq, :len(starts)] = torch.as_tensor(np.array(starts, np.int32))
        t["n_starts"][seq] = len(starts)
    if rows is not None:
        h = np.stack([r.h_last for r in rows]).astype(np.float32)
        t["h_last"][seq, :len(rows)] = torch.as_tensor(h)


def own_topk(z, k=10):
    return np.lexsort((np.arange(len(z)), -z))[:k]


def check_rows(rt, s, exp, rows, lg_call, mine, dr, branch_map, tol, tally,
               forced=None):
    """Per-row checks of one expansion for sequence s; returns whether every
    bucket equals the oracle's (then the tree's shape must too).  With
    ``forced`` (the row buckets both sides were given) the buckets must
    equal it exactly."""
    d = rt.dout
    lg = lg_call[mine]
    e = rel_err(lg, exp["logits"])
    tally.worst_logit = max(tally.worst_logit, float(e.max()))
    assert e.max() < tol, (s, e.max())
    exact = True
    rank_w = np.asarray(dr.rank_w, np.float64)
    rank_b = np.asarray(dr.rank_b, np.float64)
    for i in range(exp["R"]):
        o = exp["base"] + i
        r = rows[o]
        zg, zr = lg[i].astype(np.float64), r.logits
        E = float(np.abs(zg - zr).max())
        ids = host(d["topk_id"][s, o])
        # the device's top-k is its own logits' top-k (drafter ids, reported
        # as target ids), values copied exactly
        own = own_topk(lg[i])
        assert list(ids) == list(dr.to_target(own)), (s, o)
        assert np.array_equal(host(d["topk_logit"][s, o]), lg[i][own]), (s, o)
        lse_own = np.logaddexp.reduce(zg)
        assert abs(float(d["lse"][s, o]) - lse_own) < 1e-3 * max(1, abs(lse_own))
        # valid under the oracle's logits up to 2E
        zs = np.sort(zr)[::-1]
        assert len(set(ids.tolist())) == len(ids)
        assert np.all(np.abs(zr[own] - zs[:len(own)]) <= 2 * E + 1e-6), (s, o)
        # psi, h^(L)
        # psi: log-probabilities, gaps and p1 move by at most 2E each; the
        # entropy by at most 2E (H + 1)
        pg = host(d["psi"][s, o]).astype(np.float64)
        bound = np.full(len(pg), 4 * E + 1e-3)
        bound[-1] = 4 * E * (abs(r.psi[-1]) + 1) + 1e-3
        assert np.all(np.abs(pg - r.psi) <= bound), (s, o, pg - r.psi)
        hg = host(rt.tree["h_last"][s, o]).astype(np.float64)
        assert rel_err(hg, r.h_last) < tol, (s, o)
        # bucket: the device's is the argmax of the scores of its own h, psi;
        # against the oracle's up to twice the score error
        sg = rank_w @ np.concatenate([hg, pg]) + rank_b
        bg = int(d["bucket"][s, o])
        es = float(np.abs(sg - r.scores).max())
        if forced is not None:
            want = min(max(int(forced[o]), 0), 3)
            assert bg == want and r.bucket == want, (s, o, bg, r.bucket)
        else:
            top2 = np.sort(sg)[::-1]
            if bg != int(np.argmax(sg)):
                assert top2[0] - sg[bg] < 1e-3 * max(1.0, abs(top2[0])), (s, o)
            if bg != r.bucket:
                assert r.scores[r.bucket] - r.scores[bg] <= 2 * es + 1e-4, (s, o)
        assert int(d["branch"][s, o]) == branch_map[bg]
        b = max(branch_map[bg], r.branch)
        ok = bg == r.bucket and list(ids[:b]) == list(r.topk[:b])
        tally.rows += 1
        tally.rows_exact += ok
        exact &= bg == r.bucket
    return exact


def check_tree_exact(rt, s, tree, rows, lo, hi, tol_cum):
    """Nodes lo..hi-1 of the device tree: the shape (parents, depths, rows,
    ranks, ancestor bits) equals the oracle's exactly; every token is the
    device's own top-k id of its row and rank, and equals the oracle's token
    wherever the device's top-k agrees with the oracle's there."""
    t = rt.tree
    assert int(t["n_nodes"][s]) == hi, (s, int(t["n_nodes"][s]), hi)
    nodes = tree.nodes[lo:hi]
    for f in ("parent", "depth", "row", "rank"):
        assert list(host(t[f][s, lo:hi])) == [getattr(x, f) for x in nodes], (s, f)
    tok = host(t["token"][s, lo:hi])
    for j, x in enumerate(nodes):
        gid = host(rt.dout["topk_id"][s, x.row])
        assert tok[j] == gid[x.rank - 1], (s, lo + j)
        if gid[x.rank - 1] == rows[x.row].topk[x.rank - 1]:
            assert tok[j] == x.token, (s, lo + j)
    cum = host(t["cum_logp"][s, lo:hi]).astype(np.float64)
    assert np.all(np.abs(cum - [x.cum_logp for x in nodes]) <= tol_cum), s
    anc = host(t["anc"][s, :hi]).view(np.uint32)
    assert np.array_equal(anc[lo:hi], _anc_words(tree, hi, anc.shape[-1])[lo:hi]), s


def run_and_compare(rt, seqs, w, tgt, dr, tol, tally, log=print,
                    forced=None, deep_tol=None):
    """Drive one device iteration over all sequences, comparing the sampled
    ones; ``seqs`` maps seq -> (state before, state after, record, drafted
    tree).  The device's state for those sequences must equal the 'before'
    state when called.  ``forced``: [n_seqs][row_cap] buckets both sides
    were given, or None.  ``deep_tol`` (default ``tol``) bounds the outputs
    that went through the target's decoder stack: verify logits, taps, the
    next condition taps and the committed target K/V."""
    deep_tol = tol if deep_tol is None else deep_tol
    bmap = tuple(w.branch_map)
    for m in range(1, w.M + 1):
        log(f"expand {m}")
        rt.expand(m, want_logits=True)
        torch.cuda.synchronize()
        n_call = int(rt.dout["n_call"][0])
        cseq = host(rt.dout["call_seq"])[:n_call]
        crow = host(rt.dout["call_row"])[:n_call]
        lg = host(rt.dout["logits"])[:n_call]
        assert np.isfinite(lg).all()
        for s, (_, _, rec, drafted) in seqs.items():
            exps = rec["expansions"]
            mine = np.nonzero(cseq == s)[0]
            if m > len(exps):
                assert len(mine) == 0
                continue
            exp = exps[m - 1]
            assert len(mine) == exp["R"], (s, m, len(mine), exp["R"])
            assert list(crow[mine]) == list(range(exp["base"],
                                                  exp["base"] + exp["R"]))
            exact = check_rows(rt, s, exp, rec["rows"], lg, mine, dr, bmap,
                               tol, tally,
                               None if forced is None else forced[s])
            lo = exp["first_new"]
            hi = exps[m]["first_new"] if m < len(exps) else len(drafted)
            nxt = [sp.node for sp in exps[m]["starts"]] if m < len(exps) else []
            if exact:
                tally.calls_exact += 1
                E = float(np.abs(lg[mine] - exp["logits"]).max())
                check_tree_exact(rt, s, drafted, rec["rows"], lo, hi,
                                 4 * E * (m * w.K) + 1e-3)
                if m < w.M:
                    got = list(host(rt.tree["starts"][s, :int(rt.tree["n_starts"][s])]))
                    if got != nxt:
                        assert len(got) == len(nxt), (s, got, nxt)
                        for a, b in zip(got, nxt):
                            ca = drafted.nodes[a].cum_logp
                            cb = drafted.nodes[b].cum_logp
                            assert a == b or abs(ca - cb) <= 4 * E * w.K * m + 1e-3
            else:
                tally.calls_excused += 1
            # the next call starts from the oracle's state
            inject_tree(rt, s, drafted, hi, nxt if m < w.M else [],
                        rec["rows"])
    # verification of the oracle's (planted) tree
    for s, (_, _, rec, _) in seqs.items():
        inject_tree(rt, s, rec["tree"], len(rec["tree"]))
    log("verify")
    rt.verify(want_logits=True)
    torch.cuda.synchronize()
    n_nodes = host(rt.tree["n_nodes"])
    offs = np.concatenate([[0], np.cumsum(n_nodes)])
    for s, (_, _, rec, _) in seqs.items():
        n = len(rec["tree"])
        vl = host(rt.vout["logits"][offs[s]:offs[s] + n]).astype(np.float64)
        e = rel_err(vl, rec["verify_logits"])
        tally.worst_verify = max(tally.worst_verify, float(e.max()))
        assert e.max() < deep_tol, (s, e.max())
        g = host(rt.vout["argmax"][s, :n])
        for j in range(n):
            assert g[j] == int(np.argmax(vl[j])), (s, j)
            z = rec["verify_logits"][j]
            E = np.abs(vl[j] - z).max()
            assert z.max() - z[g[j]] <= 2 * E + 1e-6, (s, j)
        tap = host(rt.vout["taps"][s, :n]).reshape(n * 3, -1)
        assert rel_err(tap, rec["taps"].reshape(n * 3, -1)).max() < deep_tol, s
        rt.vout["argmax"][s, :n] = torch.as_tensor(
            np.asarray(rec["greedy"], np.int32))
    log("accept, commit")
    rt.accept()
    rt.commit()
    torch.cuda.synchronize()
    for s, (before, after, rec, _) in seqs.items():
        a = int(rt.aout["n_accepted"][s])
        assert a == len(rec["path"]), (s, a, rec["path"])
        assert list(host(rt.aout["path"][s, :a])) == rec["path"]
        assert int(rt.aout["bonus"][s]) == rec["bonus"]
        # verifier-derived signal: the device recomputes the bonus logit from
        # the row's cached h^(L) (bf16 operand, fp32 sums) over its own lse
        rg, rr = float(rt.aout["r_reject"][s]), rec["r_reject"]
        if rr is None:
            assert rg == -1.0, (s, rg)
        else:
            assert abs(rg - rr) <= 5e-2 * rr + 1e-7, (s, rg, rr)
        assert int(rt.T[s]) == after.T and int(rt.root[s]) == after.root
        assert rel_err(host(rt.cond_taps[s]), after.cond_taps).max() < deep_tol
        T0, n = before.T, after.T - before.T
        for which, ref in (("target", after.tkv), ("drafter", after.dkv)):
            k, v = rt.read_cache(which, s, n, T0)
            bound = deep_tol if which == "target" else tol
            for layer in range(len(ref.k)):
                for got, want in ((k[layer], ref.k[layer][T0:]),
                                  (v[layer], ref.v[layer][T0:])):
                    assert rel_err(got.reshape(n, -1),
                                   want.reshape(n, -1)).max() < bound, (s, which)
