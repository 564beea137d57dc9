"""GPU parity over a seeded sweep of random configurations on the tiny fp32
model (2-layer target, d 256): block depth K, block count M, starts per
block B_max, tree budget, number of sequences, prompt lengths (from one
token up, across page boundaries), the bucket -> branching map (entries
0..10, so some buckets add no tokens), one or two drafter layers, and the
bucket mode (the rank head's own argmax or paper-frequency draws).  Each
configuration runs one iteration compared call by call with the oracle
(teacher forcing oracle -> device, see parity_checks; fp32 tolerance 1e-4
relative, discrete outputs margin-aware), the committed prefix seeded
random K/V.  The draws are fixed by the case seed, so a failure names its
configuration and reproduces."""
import numpy as np
import pytest

import synth

from gpu_harness import inject, models, runtime
from parity_checks import Tally, oracle_iteration, run_and_compare
from test_gpu_configs import synthetic_state

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]
TOL = 1e-4
N_CASES = 24


def sweep_workload(seed: int):
    """A random valid configuration (the limits sb_create enforces: row
    capacity K + (M - 1) B_max K <= 512, B_max <= 64, budget <= 512) and its
    bucket mode."""
    rng = np.random.default_rng([seed, 2605])
    K = int(rng.integers(1, 9))
    M = int(rng.integers(1, 5))
    B_max = int(rng.integers(1, 17))
    while K + (M - 1) * B_max * K > 512:
        B_max -= 1
    budget = int(rng.integers(2, 201))
    n_seqs = int(rng.integers(1, 7))
    lo = int(rng.integers(1, 41))
    hi = int(rng.integers(lo, 301))
    bmap = tuple(int(v) for v in rng.integers(0, 11, 4))
    layers = int(rng.integers(1, 3))
    paper = bool(rng.integers(0, 2))
    w = synth.Workload(f"sweep{seed}-fp32", "f32", synth.TINY, layers, K=K,
                       M=M, B_max=B_max, budget=budget, n_seqs=n_seqs,
                       prompt_len=(lo, hi), branch_map=bmap)
    return w, paper


def log(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_configuration(seed):
    w, paper = sweep_workload(seed)
    tag = (f"[sweep {seed}: K {w.K} M {w.M} B_max {w.B_max} budget "
           f"{w.budget} seqs {w.n_seqs} prompts {w.prompt_len} map "
           f"{w.branch_map} drafter layers {w.drafter_layers} "
           f"{'paper' if paper else 'natural'} buckets]")
    log(f"{tag} models")
    weights, tgt, dr = models(w)
    lens = synth.prompt_lengths(w)
    states = [synthetic_state(w, tgt, dr, s, int(lens[s]), 100 + seed)
              for s in range(w.n_seqs)]
    rt = runtime(w, weights,
                 max_pages=(int(max(lens)) + w.M * w.K + 16) // 16 + 1)
    for s, st in enumerate(states):
        inject(rt, s, st)
    forced = (synth.paper_buckets(seed, 0, w.n_seqs, rt.row_cap)
              if paper else None)
    if forced is not None:
        import torch
        rt.set_buckets(torch.as_tensor(forced).to(rt.dev))
    seqs = {}
    for s in range(w.n_seqs):
        depth = (w.K + 1 + 2 * s + seed) % (w.M * w.K + 1)
        seqs[s] = (states[s],) + oracle_iteration(
            tgt, dr, states[s], w, depth,
            None if forced is None else forced[s])
    log(f"{tag} oracle trees {[len(seqs[s][3]) for s in seqs]} nodes")
    tally = Tally()
    run_and_compare(rt, seqs, w, tgt, dr, TOL, tally,
                    log=lambda m: log(f"[sweep {seed}] {m}"), forced=forced)
    log(f"[sweep {seed}] {tally}")
    if forced is not None:
        rt.set_buckets(None)
    assert tally.rows == sum(sum(e["R"] for e in seqs[s][2]["expansions"])
                             for s in seqs)


BF16_SHAPE = synth.ModelShape(2, 512, 8, 2, 128, 1536, 4096)
N_BF16 = 12


def sweep_workload_bf16(seed: int):
    """A random bf16 configuration at d 512 (grouped-query attention, four
    query heads per KV head, head_dim 128): up to 24 sequences (from 16 the
    32x32 attention kernel takes over), budgets up to 160, so that the
    projections run few- and many-row tiles (1-, 2- and 4-fragment rows);
    the oracle samples up to three sequences."""
    rng = np.random.default_rng([seed, 512])
    K = int(rng.integers(1, 9))
    M = int(rng.integers(1, 4))
    B_max = int(rng.integers(1, 17))
    while K + (M - 1) * B_max * K > 512:
        B_max -= 1
    budget = int(rng.integers(2, 161))
    n_seqs = int(rng.integers(1, 25))
    lo = int(rng.integers(1, 41))
    hi = int(rng.integers(lo, 301))
    bmap = tuple(int(v) for v in rng.integers(0, 11, 4))
    paper = bool(rng.integers(0, 2))
    w = synth.Workload(f"sweep{seed}-bf16", "bf16", BF16_SHAPE, 1, K=K, M=M,
                       B_max=B_max, budget=budget, n_seqs=n_seqs,
                       prompt_len=(lo, hi), branch_map=bmap)
    sample = tuple(sorted({0, n_seqs // 2, n_seqs - 1}))
    return w, paper, sample


@pytest.mark.parametrize("seed", range(N_BF16))
def test_random_configuration_bf16(seed):
    """The same at bf16 (tolerance 2e-2 relative, discrete outputs
    margin-aware)."""
    import torch
    w, paper, sample = sweep_workload_bf16(seed)
    tag = (f"[bf16 sweep {seed}: K {w.K} M {w.M} B_max {w.B_max} budget "
           f"{w.budget} seqs {w.n_seqs} prompts {w.prompt_len} map "
           f"{w.branch_map} {'paper' if paper else 'natural'} buckets]")
    log(f"{tag} models")
    weights, tgt, dr = models(w)
    lens = synth.prompt_lengths(w)
    states = [synthetic_state(w, tgt, dr, s, int(lens[s]), 200 + seed)
              for s in range(w.n_seqs)]
    rt = runtime(w, weights,
                 max_pages=(int(max(lens)) + w.M * w.K + 16) // 16 + 1)
    for s, st in enumerate(states):
        inject(rt, s, st)
    forced = (synth.paper_buckets(seed, 0, w.n_seqs, rt.row_cap)
              if paper else None)
    if forced is not None:
        rt.set_buckets(torch.as_tensor(forced).to(rt.dev))
    seqs = {}
    for s in sample:
        depth = (w.K + 1 + 2 * s + seed) % (w.M * w.K + 1)
        seqs[s] = (states[s],) + oracle_iteration(
            tgt, dr, states[s], w, depth,
            None if forced is None else forced[s])
    log(f"{tag} oracle trees {[len(seqs[s][3]) for s in seqs]} nodes "
        f"(sequences {sample})")
    tally = Tally()
    run_and_compare(rt, seqs, w, tgt, dr, 2e-2, tally,
                    log=lambda m: log(f"[bf16 sweep {seed}] {m}"),
                    forced=forced)
    log(f"[bf16 sweep {seed}] {tally}")
    if forced is not None:
        rt.set_buckets(None)
    assert tally.rows == sum(sum(e["R"] for e in seqs[s][2]["expansions"])
                             for s in seqs)
