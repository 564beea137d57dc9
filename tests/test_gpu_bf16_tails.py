"""GPU parity where the projection widths are not multiples of the GEMM
workgroup span: vocabulary 4032 (= 63 x 64, so the last weight tile of the
LM heads is partly past the matrix) with two sequences and a 96-node tree
budget (192 verify rows: 128-row activation tiles with 64 weight rows per
wave), and 100-token prompts prefilled in 64-row chunks.  Oracle prefill,
then one iteration compared call by call on the oracle's inputs for both
sequences (see parity_checks)."""
import pytest

import synth
from oracle import specdec

from gpu_harness import inject, models, runtime
from parity_checks import Tally, oracle_iteration, run_and_compare

pytestmark = pytest.mark.gpu
TOL = 2e-2

SHAPE = synth.ModelShape(2, 512, 8, 2, 128, 1536, 4032)
W = synth.Workload("tails-bf16", "bf16", SHAPE, 1, K=4, M=2, B_max=8,
                   budget=96, n_seqs=2, prompt_len=(100, 100))


def test_iteration_calls_width_tails():
    weights, tgt, dr = models(W)
    prompts = synth.prompts(W)
    states = [specdec.prefill(tgt, dr, pr) for pr in prompts]
    rt = runtime(W, weights, max_pages=24, prefill_chunk=64)
    for s, st in enumerate(states):
        inject(rt, s, st)
    seqs = {}
    for s, st in enumerate(states):
        seqs[s] = (st,) + oracle_iteration(tgt, dr, st, W, 2 + 3 * s)
    tally = Tally()
    run_and_compare(rt, seqs, W, tgt, dr, TOL, tally,
                    log=lambda m: print(m, flush=True))
    print(tally, flush=True)
    assert tally.rows == sum(sum(e["R"] for e in seqs[s][2]["expansions"])
                             for s in seqs)


def test_prefill_chunks_width_tails():
    """Device prefill in 64-row chunks against the oracle's prefill."""
    import numpy as np
    import torch
    from gpu_harness import host, rel_err
    weights, tgt, dr = models(W)
    prompts = synth.prompts(W)
    rt = runtime(W, weights, max_pages=24, prefill_chunk=64)
    rt.prefill(prompts)
    torch.cuda.synchronize()
    for s, pr in enumerate(prompts):
        st = specdec.prefill(tgt, dr, pr)
        assert int(rt.T[s]) == st.T
        k, v = rt.read_cache("target", s, st.T)
        for layer in range(SHAPE.n_layers):
            assert rel_err(k[layer].reshape(st.T, -1),
                           st.tkv.k[layer].reshape(st.T, -1)).max() < TOL
            assert rel_err(v[layer].reshape(st.T, -1),
                           st.tkv.v[layer].reshape(st.T, -1)).max() < TOL
        assert rel_err(host(rt.cond_taps[s]), st.cond_taps).max() < TOL
        assert np.isfinite(host(rt.cond_taps[s])).all()
