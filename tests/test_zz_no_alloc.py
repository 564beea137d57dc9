"""The allocation-free stochastic acceptance (sb_accept_sample_noalloc,
static scratch) against the workspace entry point sb_accept_sample, through
the C ABI: identical paths, accepted counts, bonus tokens and signals on the
same trees, logits and uniforms, for two calls in a row (the second with
fewer sequences and smaller trees, so the scratch holds the first call's
larger contents), in both call orders.  The vocabulary spans eight 16384-token
statistics tiles."""
import numpy as np
import pytest
import torch

import synth

from gpu_harness import host, runtime
from parity_checks import inject_tree
from test_gpu_sampling import random_tree, synthetic_logits

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]


def _set_inputs(rt, rng, n_seqs, budget, V, cap, max_nodes):
    rows = []
    for s in range(n_seqs):
        t = random_tree(rng, min(budget, max_nodes), cap, V)
        inject_tree(rt, s, t, len(t))
        rows.append(synthetic_logits(rng, t, V))
    z = np.concatenate(rows)
    rt.vout["logits"][:len(z)] = torch.as_tensor(z)
    ua = torch.as_tensor(rng.random((rt.S, budget)).astype(np.float32))
    ub = torch.as_tensor(rng.random((rt.S, budget)).astype(np.float32))
    return ua.to(rt.dev), ub.to(rt.dev)


def _result(rt, n_seqs):
    torch.cuda.synchronize()
    return {k: host(rt.aout[k][:n_seqs]).copy()
            for k in ("path", "n_accepted", "bonus", "r_reject")}


def test_noalloc_matches_workspace_entry_point():
    w = synth.with_layers(synth.WORKLOADS["llama3-8b-k4"], 1)
    V, budget, cap = w.target.vocab, w.budget, w.M * w.K
    rt = runtime(w, None, n_seqs=3)
    rt.vout["logits"] = torch.zeros(rt.S * budget, V, dtype=torch.float32,
                                    device=rt.dev)
    # (sequences, node cap, temperature): the second call is smaller
    calls = [(3, budget, 1.0), (1, 9, 0.7)]
    for order in (("ws", "noalloc"), ("noalloc", "ws")):
        for i, (n, max_nodes, temp) in enumerate(calls):
            rng = np.random.default_rng([23, i, len(order[0])])
            ua, ub = _set_inputs(rt, rng, n, budget, V, cap, max_nodes)
            print(f"[noalloc] order {order} call {i}: {n} seqs, "
                  f"<= {max_nodes} nodes, T {temp}", flush=True)
            got = {}
            for which in order:
                rt.aout["path"].fill_(-7)
                rt.aout["bonus"].fill_(-7)
                rt.accept_sample(temp, ua, ub, noalloc=(which == "noalloc"),
                                 n_seqs=n)
                got[which] = _result(rt, n)
            for k in got["ws"]:
                np.testing.assert_array_equal(got["noalloc"][k], got["ws"][k],
                                              err_msg=f"{order} call {i} {k}")
            assert (got["ws"]["bonus"] >= 0).all()
