"""A length bound below a sequence's T (sb_set_length_bound) makes tree
attention skip the committed entries past it, in every attention path: the
16-row kernel (one sequence, 60 nodes over a 1024-entry prefix), the 32x32
kernel with balanced splits (one sequence, 128 nodes over 4096 entries) and
with fixed splits (16 ragged sequences).

With the bound B in place, the committed target K/V entries B.. of every
sequence are overwritten with NaN: verification must then give bit-identical
logits, argmax and taps, all finite (an entry read past the bound would
carry the NaN into them).  Against verification under a bound above every
T, the logits of a sequence whose prefix is longer than B must change (by
more than 2e-2 relative: a few hundred keys of random K/V are dropped),
those of the others must not (within 2e-2: the bound changes the split plan,
hence the summation order).  Weights are generated on the device (one target
layer); no oracle is involved, the property is the device's own.
"""
import numpy as np
import pytest
import torch

import synth
from gpu_harness import rel_err
from paper_2605_07243_amd.runtime import Runtime

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]

CASES = {
    # name: (workload, bound below the prompts' lengths)
    "16-row": ("llama3-8b-k4", 800),
    "32x32-balanced": ("llama3-8b-k8-long", 3500),
    "32x32-fixed": ("llama3-8b-batch16-paged", 1200),
}


def _verify(rt):
    rt.verify(want_logits=True)
    torch.cuda.synchronize()
    return {k: rt.vout[k].clone() for k in ("logits", "argmax", "taps")}


@pytest.mark.parametrize("name", list(CASES))
def test_entries_past_the_bound_are_skipped(name):
    wname, bound = CASES[name]
    w = synth.with_layers(synth.WORKLOADS[wname], 1)
    print(f"[{name}] runtime", flush=True)
    rt = Runtime(w, None, seed=3)
    rt.prefill(synth.prompts(w))
    for m in range(1, w.M + 1):
        rt.expand(m)
    torch.cuda.synchronize()
    T = rt.T.cpu().numpy()
    assert (T > bound).any()
    print(f"[{name}] T {sorted(T.tolist())[:4]}... bound {bound}", flush=True)
    rt.set_length_bound(int(T.max()) + 1)
    full = _verify(rt)
    rt.set_length_bound(bound)
    cut = _verify(rt)
    s = w.target
    for seq in np.nonzero(T > bound)[0]:
        n = int(T[seq]) - bound
        nan = np.full((1, n, s.n_kv_heads, s.head_dim), np.nan, np.float32)
        rt.write_cache("target", int(seq), nan, nan, bound)
    torch.cuda.synchronize()
    print(f"[{name}] verify with NaN past the bound", flush=True)
    poisoned = _verify(rt)
    for k in cut:
        assert torch.equal(poisoned[k], cut[k]), k
    # verify logits are in call-row order: each sequence's nodes in turn
    nodes = rt.tree["n_nodes"].cpu().numpy().astype(np.int64)
    first = np.concatenate([[0], np.cumsum(nodes)])
    for seq in range(w.n_seqs):
        rows = slice(int(first[seq]), int(first[seq + 1]))
        assert torch.isfinite(poisoned["logits"][rows]).all(), seq
        err = float(rel_err(cut["logits"][rows].cpu().numpy(),
                            full["logits"][rows].cpu().numpy()).max())
        print(f"[{name}] seq {seq} T {int(T[seq])}: bound moves logits by "
              f"{err:.2e}", flush=True)
        if T[seq] > bound:
            assert err > 2e-2, (seq, err)
        else:
            assert err <= 2e-2, (seq, err)
    rt.set_length_bound(int(T.max()) + 1)
