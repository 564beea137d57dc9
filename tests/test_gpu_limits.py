"""GPU parity at the configuration's limits, on the tiny fp32 model (2-layer
target, d 256) so that the oracle recomputes every call:

* a 512-node tree budget (sixteen ancestor words per node) with the row
  capacity K + (M - 1) B_max K at its limit of 512 (K = 8, M = 2, B_max =
  63: block 2 runs up to 504 rows, within the attachment's 512-row stage),
  for three sequences with ragged prompts across page boundaries, once with
  buckets forced from the paper-frequency draws and once as the uniform
  fixed-8 tree (every row b1, eight tokens per row: block 1 puts 57
  next-block starts forward and block 2 fills the budget);
* B_max = 64 starts per block, the start limit (K = 7, uniform fixed-10
  tree: ten tokens per row, the branching maximum, so block 1 puts exactly
  64 starts forward);
* 64 sequences, the per-call maximum, with small trees; the oracle recomputes
  four of them while the device runs all;
* the shortest prompts and page edges: prompts of 1, 2, 16, 17 and 33 tokens
  through the device prefill (against the oracle's) and one iteration;
* fp32 with 128-wide heads (two heads, d 256), where the attention launch
  takes its fallback shapes: one q-tile of queries per KV head (two-wave
  workgroups whose second wave has no queries) and, with 16 sequences x 2
  KV heads and 144-node trees, one q-tile per wave where bf16 takes two.

The committed prefix is seeded random K/V (as at the benchmark shapes), one
iteration is compared call by call with teacher forcing (see parity_checks),
fp32 tolerance 1e-4 relative, discrete outputs margin-aware."""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import specdec

from gpu_harness import host, inject, models, rel_err, runtime
from parity_checks import Tally, oracle_iteration, run_and_compare
from test_gpu_configs import synthetic_state

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]
TOL = 1e-4

BIG_TREE = synth.Workload("limits-fp32", "f32", synth.TINY, 1, K=8, M=2,
                          B_max=63, budget=512, n_seqs=3,
                          prompt_len=(20, 300))
WIDE = synth.Workload("wide-fp32", "f32", synth.TINY, 1, K=7, M=2,
                      B_max=64, budget=512, n_seqs=2, prompt_len=(40, 260))
MANY_SEQS = synth.Workload("many-seqs-fp32", "f32", synth.TINY, 1, K=4, M=2,
                           B_max=4, budget=16, n_seqs=64,
                           prompt_len=(10, 200))

HD128 = synth.ModelShape(2, 256, 2, 2, 128, 512, 1024)
HD128_ONE_QTILE = synth.Workload("hd128-fp32", "f32", HD128, 1, K=4, M=2,
                                 B_max=4, budget=16, n_seqs=2,
                                 prompt_len=(40, 90))
HD128_MANY = synth.Workload("hd128-16seq-fp32", "f32", HD128, 1, K=4, M=2,
                            B_max=8, budget=144, n_seqs=16,
                            prompt_len=(20, 120))

CASES = {
    # name: (workload, uniform fixed-k tree (0: paper-frequency buckets; -1:
    # the rank head's own), sequences the oracle runs)
    "budget512-paper": (BIG_TREE, 0, None),
    "budget512-uniform8": (BIG_TREE, 8, None),
    "bmax64-uniform10": (WIDE, 10, None),
    "64-sequences": (MANY_SEQS, -1, (0, 21, 42, 63)),
    "f32-head-dim-128-one-qtile": (HD128_ONE_QTILE, -1, None),
    "f32-head-dim-128-16-sequences": (HD128_MANY, 0, (0, 7, 15)),
}


def log(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("name", list(CASES))
def test_iteration_at_limits(name):
    w, k, sample = CASES[name]
    if k > 0:
        w = synth.uniform_tree(w, k)
    weights, tgt, dr = models(w)
    lens = synth.prompt_lengths(w)
    sample = sample or tuple(range(w.n_seqs))
    log(f"[{name}] prompts {sorted(lens.tolist())[:6]}..., runtime")
    states = [synthetic_state(w, tgt, dr, s, int(lens[s]), 11)
              for s in range(w.n_seqs)]
    rt = runtime(w, weights,
                 max_pages=(int(max(lens)) + w.M * w.K + 16) // 16 + 1)
    for s, st in enumerate(states):
        inject(rt, s, st)
    forced = (synth.uniform_buckets(w.n_seqs, rt.row_cap) if k > 0 else
              synth.paper_buckets(7, 0, w.n_seqs, rt.row_cap) if k == 0 else
              None)
    if forced is not None:
        rt.set_buckets(torch.as_tensor(forced).to(rt.dev))
    seqs = {}
    for s in sample:
        depth = (w.K + 2 + 3 * s) % (2 * w.K + 1)
        log(f"[{name}] oracle seq {s} (T {states[s].T}, planted depth {depth})")
        seqs[s] = (states[s],) + oracle_iteration(
            tgt, dr, states[s], w, depth,
            None if forced is None else forced[s])
    sizes = [len(seqs[s][3]) for s in seqs]
    starts = [max(len(e["starts"]) for e in seqs[s][2]["expansions"])
              for s in seqs]
    log(f"[{name}] oracle trees {sizes} nodes, most starts per block {starts}")
    if k > 0:
        # the limits are reached: full trees (ancestor bits in word 15) and
        # as many starts as the block's rows put forward, up to B_max
        assert max(sizes) == 512
        assert max(starts) == min(w.B_max, w.K * (k - 1) + 1)
    tally = Tally()
    run_and_compare(rt, seqs, w, tgt, dr, TOL, tally,
                    log=lambda m: log(f"[{name}] {m}"), forced=forced)
    log(f"[{name}] {tally}")
    if forced is not None:
        rt.set_buckets(None)
    assert tally.rows == sum(sum(e["R"] for e in seqs[s][2]["expansions"])
                             for s in seqs)


EDGE = synth.Workload("edge-prompts-fp32", "f32", synth.TINY, 1, K=4, M=3,
                      B_max=4, budget=32, n_seqs=5, prompt_len=(1, 33))


def test_short_and_page_edge_prompts():
    """Prompts of 1, 2, 16, 17 and 33 tokens: a one-token prompt commits one
    entry (its drafter entry conditioned on zero taps, reading R2) and the
    root is the target's next token; 16 and 17 end on and just past a page
    boundary.  Device prefill against the oracle's (caches, root, condition
    taps), then one iteration compared call by call."""
    w = EDGE
    weights, tgt, dr = models(w)
    lens = [1, 2, 16, 17, 33]
    prompts = synth.prompts(w, lengths=lens)
    states = [specdec.prefill(tgt, dr, pr) for pr in prompts]
    rt = runtime(w, weights, max_pages=8)
    log("[edge] prefill")
    rt.prefill(prompts)
    torch.cuda.synchronize()
    for s, st in enumerate(states):
        assert int(rt.T[s]) == st.T, s
        assert int(rt.root[s]) == st.root, s
        assert rel_err(host(rt.cond_taps[s]), st.cond_taps).max() < TOL, s
        for which, kv, layers in (("target", st.tkv, w.target.n_layers),
                                  ("drafter", st.dkv, w.drafter_layers)):
            k, v = rt.read_cache(which, s, st.T)
            for layer in range(layers):
                for got, ref in ((k, kv.k), (v, kv.v)):
                    assert rel_err(got[layer].reshape(st.T, -1),
                                   ref[layer].reshape(st.T, -1)).max() < TOL, \
                        (s, which, layer)
    for s, st in enumerate(states):
        inject(rt, s, st)
    seqs = {}
    for s, st in enumerate(states):
        seqs[s] = (st,) + oracle_iteration(tgt, dr, st, w, 2 + s)
    tally = Tally()
    run_and_compare(rt, seqs, w, tgt, dr, TOL, tally,
                    log=lambda m: log(f"[edge] {m}"))
    log(f"[edge] {tally}")
    assert tally.rows == sum(sum(e["R"] for e in seqs[s][2]["expansions"])
                             for s in seqs)
