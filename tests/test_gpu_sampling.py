"""GPU parity of stochastic tree verification (sb_accept_sample) against the
oracle's walk, on the same trees, target logits and uniforms.

Trees are synthetic (random parents within the depth bound M K, tokens from a
small pool so that siblings sometimes repeat a token), the logits are random
with the children's tokens boosted so that acceptances are frequent, and the
uniforms come from a seeded generator; the device writes every input's
float32 value, and the oracle reads the same float32 values.  Accepted paths
must be identical wherever every acceptance test of the oracle's walk has a
margin |u - r(x)| above 1e-4 (the float32 error of r is ~1e-6); those closer
are excused and counted.  The bonus token must be identical where the
oracle's bonus target lies farther than CDF_TOL (relative to the residual
total) from the cumulative-mass boundaries of its token: the device sums the
masses in float64, so its boundaries carry only the float32 error of the
individual probabilities (~5e-7 relative each).  Closer than that, the
device's token must still be one whose boundaries lie within CDF_TOL of the
target (with 128256 tokens of ~1e-5 mass each this case is common).  Two workloads: the
tiny fp32 one (vocabulary 1024, budget 32) and the 8B-shaped bf16 one with
two sequences (vocabulary 128256, budget 60), so that the call-row offsets
of a second sequence are exercised.
"""
import numpy as np
import pytest
import torch

import synth
from oracle.sampling import accept_sample, target_probs
from oracle.tree import DraftTree

from gpu_harness import host, runtime
from parity_checks import inject_tree

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]
MARGIN = 1e-4
CDF_TOL = 2e-6


def random_tree(rng, budget, max_depth, vocab):
    n = int(rng.integers(1, budget + 1))
    pool = rng.choice(vocab, size=12, replace=False)
    t = DraftTree(int(rng.integers(vocab)), budget)
    for _ in range(1, n):
        cands = [i for i in range(len(t)) if t.nodes[i].depth < max_depth]
        # favour recent nodes so that paths get deep
        par = cands[max(0, len(cands) - 1 - int(rng.exponential(3.0)))]
        t.add(int(rng.choice(pool)), par, 0, 1, 0.0)
    return t


def synthetic_logits(rng, tree, vocab):
    z = rng.standard_normal((len(tree), vocab)).astype(np.float32)
    for n in range(len(tree)):
        for c in tree.children(n):
            z[n, tree.nodes[c].token] += np.float32(rng.uniform(2.0, 11.0))
    return z


@pytest.mark.parametrize("wname,n_seqs", [("tiny-fp32", 1),
                                          ("llama3-8b-k4", 2)])
def test_accept_sample_matches_oracle(wname, n_seqs):
    w = synth.with_layers(synth.WORKLOADS[wname], 1)
    V, budget, cap = w.target.vocab, w.budget, w.M * w.K
    print(f"[{wname}] runtime", flush=True)
    rt = runtime(w, None, n_seqs=n_seqs)
    rt.vout["logits"] = torch.zeros(n_seqs * budget, V, dtype=torch.float32,
                                    device=rt.dev)
    exact = excused = accepted = bonus_exact = 0
    trials = 12 if V > 10_000 else 40
    for trial in range(trials):
        rng = np.random.default_rng([11, trial])
        temperature = (1.0, 0.7, 1.6)[trial % 3]
        trees, zs = [], []
        for s in range(n_seqs):
            t = random_tree(rng, budget, cap, V)
            trees.append(t)
            zs.append(synthetic_logits(rng, t, V))
            inject_tree(rt, s, t, len(t))
        rows = np.concatenate(zs)
        rt.vout["logits"][:len(rows)] = torch.as_tensor(rows)
        ua = rng.random((n_seqs, budget)).astype(np.float32)
        ub = rng.random((n_seqs, budget)).astype(np.float32)
        print(f"[{wname}] trial {trial} T {temperature} nodes "
              f"{[len(t) for t in trees]}", flush=True)
        rt.accept_sample(temperature, torch.as_tensor(ua).to(rt.dev),
                         torch.as_tensor(ub).to(rt.dev))
        torch.cuda.synchronize()
        for s, t in enumerate(trees):
            ref = accept_sample(t, zs[s].astype(np.float64), temperature,
                                ua[s].astype(np.float64),
                                ub[s].astype(np.float64))
            a = int(rt.aout["n_accepted"][s])
            path = list(host(rt.aout["path"][s, :a]))
            bonus = int(rt.aout["bonus"][s])
            # always: a valid walk (parent -> child edges from the root)
            prev = 0
            for n in path:
                assert t.nodes[n].parent == prev, (trial, s, path)
                prev = n
            assert 0 <= bonus < V
            if ref["test_margin"] <= MARGIN:
                excused += 1
                continue
            assert path == ref["path"], (trial, s, path, ref["path"])
            exact += 1
            accepted += len(path)
            if ref["cdf_margin"] > CDF_TOL:
                assert bonus == ref["bonus"], (trial, s, bonus, ref["bonus"])
                bonus_exact += 1
            else:
                # valid draw: the target lies within CDF_TOL of the device
                # token's interval of the oracle's residual CDF
                end = path[-1] if path else 0
                wres = target_probs(zs[s][end].astype(np.float64),
                                    temperature)
                tested = [t.nodes[c].token for c in sorted(t.children(end))]
                wres[[x for x in tested]] = 0.0
                cdf = np.cumsum(wres)
                tot = cdf[-1]
                tgt = float(ub[s][end]) * tot
                lo = cdf[bonus - 1] if bonus > 0 else 0.0
                assert wres[bonus] > 0.0, (trial, s, bonus)
                assert lo - CDF_TOL * tot <= tgt < cdf[bonus] + CDF_TOL * tot, \
                    (trial, s, bonus, ref["bonus"])
    print(f"[{wname}] paths exact {exact} excused {excused}, bonus exact "
          f"{bonus_exact}, accepted nodes {accepted}", flush=True)
    assert exact >= 0.9 * (exact + excused)
    assert accepted > exact // 4     # the walks do go down the trees
