"""Run-to-run determinism of the device path (a check for LDS races,
unordered reductions and reads of memory the call did not write).

At every benchmark workload's per-layer shape (one target layer, weights
generated on the device), the calls of one iteration (block expansions,
tree verification, acceptance) run twice from the same committed state.
Between the two runs a detour iteration with every drafter row forced into
bucket b3 (a different tree, so every scratch buffer is refilled with other
values) runs from that state too.  All outputs of the two runs, over their
valid extents, must be bit-identical; the same is checked again after a
commit.  No oracle is involved: the property is the device's own.
"""
import numpy as np
import pytest
import torch

import synth
from paper_2605_07243_amd.runtime import Runtime

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]

CASES = ["llama3-8b-k4", "llama3-8b-k8-long", "llama3-8b-batch16-paged",
         "llama3-70b-k6", "llama3-8b-paper-drafter"]


def _bits(t):
    t = t.detach().clone()
    return t.view(torch.int32) if t.dtype == torch.float32 else t


def _run(rt, w):
    """One iteration's expansions, verification and acceptance; every
    output over its valid extent (device tensors)."""
    out = {}
    for m in range(1, w.M + 1):
        rt.expand(m, want_logits=True)
        n_call = int(rt.dout["n_call"][0])
        out[f"b{m}.n_call"] = rt.dout["n_call"].clone()
        out[f"b{m}.call_row"] = _bits(rt.dout["call_row"][:n_call])
        out[f"b{m}.call_seq"] = _bits(rt.dout["call_seq"][:n_call])
        out[f"b{m}.logits"] = _bits(rt.dout["logits"][:n_call])
    t, d = rt.tree, rt.dout
    nodes = t["n_nodes"].cpu().numpy()
    rows = t["n_rows"].cpu().numpy()
    starts = t["n_starts"].cpu().numpy()
    out["n_nodes"], out["n_rows"] = t["n_nodes"].clone(), t["n_rows"].clone()
    for s in range(w.n_seqs):
        n, r = int(nodes[s]), int(rows[s])
        for f in ("token", "parent", "depth", "row", "rank", "logp",
                  "cum_logp", "anc"):
            out[f"{s}.{f}"] = _bits(t[f][s, :n])
        for f in ("row_block", "row_start", "row_k", "row_pos", "row_vis",
                  "h_last"):
            out[f"{s}.{f}"] = _bits(t[f][s, :r])
        out[f"{s}.starts"] = _bits(t["starts"][s, :int(starts[s])])
        for f in ("topk_id", "topk_logit", "lse", "psi", "bucket", "branch"):
            out[f"{s}.{f}"] = _bits(d[f][s, :r])
    rt.verify(want_logits=True)
    total = int(nodes.sum())
    out["v.logits"] = _bits(rt.vout["logits"][:total])
    for s in range(w.n_seqs):
        n = int(nodes[s])
        out[f"{s}.argmax"] = _bits(rt.vout["argmax"][s, :n])
        out[f"{s}.taps"] = _bits(rt.vout["taps"][s, :n])
    rt.accept()
    a = rt.aout["n_accepted"].cpu().numpy()
    for f in ("n_accepted", "bonus", "r_reject"):
        out[f"a.{f}"] = _bits(rt.aout[f])
    for s in range(w.n_seqs):
        out[f"{s}.path"] = _bits(rt.aout["path"][s, :int(a[s])])
    torch.cuda.synchronize()
    return out


def _same(a, b, tag):
    assert a.keys() == b.keys()
    for k in a:
        assert torch.equal(a[k], b[k]), f"{tag}: {k} differs between runs"


@pytest.mark.parametrize("name", CASES)
def test_two_runs_are_bit_identical(name):
    w = synth.with_layers(synth.WORKLOADS[name], 1)
    print(f"[{name}] runtime", flush=True)
    rt = Runtime(w, None, seed=5)
    rt.prefill(synth.prompts(w))
    detour = torch.full((w.n_seqs, rt.row_cap), 3, dtype=torch.int32,
                        device=rt.dev)
    for phase in ("after prefill", "after a commit"):
        first = _run(rt, w)
        rt.set_buckets(detour)
        other = _run(rt, w)
        rt.set_buckets(None)
        # the detour really computed something else
        assert any(not torch.equal(first[k], other[k]) for k in first
                   if k.endswith(".logits") or k.endswith(".bucket"))
        second = _run(rt, w)
        _same(first, second, f"{name} {phase}")
        print(f"[{name}] {phase}: {len(first)} outputs bit-identical "
              f"({int(first['n_nodes'].sum())} tree nodes)", flush=True)
        rt.commit()
        torch.cuda.synchronize()
