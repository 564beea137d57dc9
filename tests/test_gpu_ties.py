"""Vocabulary reductions under exact ties (tiny fp32 workload).

The drafter's and the target's LM heads repeat their rows with period P, so
every logit occurs V / P times in a row.  The top-10 of a drafter row (ties
to the smaller id, App. B's psi and the branching read it) and the greedy
arg-max of a verified node are compared with those of the device's own
logits, worked out here by sorting; lse against the same logits in fp64.
P = 8 leaves fewer distinct per-thread maxima than ten, so every logit of a
chunk is a candidate and the reduction takes its sorted-list path; P = 512
gives about twenty candidates with each value twice."""
import numpy as np
import pytest
import torch

import synth
from oracle import specdec
from oracle.model import Drafter, Target

from gpu_harness import host, inject, runtime

pytestmark = pytest.mark.gpu


def _tied(w, period):
    tw = synth.make_weights(synth.target_specs(w.target), 0, w.dtype,
                            jitter=0.1)
    dw = synth.drafter_weights(w, 0, jitter=0.1)
    for d, key in ((tw, "lm_head"), (dw, "d.lm_head")):
        rows = np.asarray(d[key])
        d[key] = np.ascontiguousarray(rows[np.arange(rows.shape[0]) % period])
    tgt = Target(tw, w.target, w.dtype, w.tap_layers)
    dr = Drafter(dw, w.target, w.dtype, w.drafter_layers, tgt.embed)
    return {**tw, **dw}, tgt, dr


def _lse(z):
    z = np.asarray(z, np.float64)
    m = z.max()
    return m + np.log(np.exp(z - m).sum())


@pytest.mark.parametrize("period", [8, 512])
def test_reductions_with_ties(period):
    w = synth.WORKLOADS["tiny-fp32"]
    weights, tgt, dr = _tied(w, period)
    prompt = synth.prompts(w)[0]
    st = specdec.prefill(tgt, dr, prompt)
    rt = runtime(w, weights, max_pages=32)
    inject(rt, 0, st)
    print(f"[ties P={period}] expand", flush=True)
    rt.expand(1, want_logits=True)
    torch.cuda.synchronize()
    d = rt.dout
    n_call = int(d["n_call"][0])
    assert n_call > 0
    rows = host(d["call_row"])[:n_call]
    lg = host(d["logits"])[:n_call]
    tied = 0
    for i, o in enumerate(rows):
        z = lg[i]
        order = sorted(range(len(z)), key=lambda v: (-z[v], v))[:10]
        assert list(host(d["topk_id"][0, o])) == order, (period, i)
        assert np.array_equal(host(d["topk_logit"][0, o]), z[order])
        assert abs(float(d["lse"][0, o]) - _lse(z)) < 1e-4 * max(1.0, abs(_lse(z)))
        tied += int(np.sum(z == z.max()) > 1)
    assert tied == n_call          # every row does tie at its maximum
    for m in range(2, w.M + 1):
        rt.expand(m)
    print(f"[ties P={period}] verify", flush=True)
    rt.verify(want_logits=True)
    torch.cuda.synchronize()
    n = int(rt.tree["n_nodes"][0])
    vl = host(rt.vout["logits"])[:n]
    am = host(rt.vout["argmax"][0, :n])
    for j in range(n):
        z = vl[j]
        assert int(am[j]) == int(np.flatnonzero(z == z.max())[0]), (period, j)
        assert np.sum(z == z.max()) > 1
