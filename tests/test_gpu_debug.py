"""Device-side range checks on caller-supplied indices (sb_set_debug,
sb_device_check).

Kernels clamp every page-table entry into 0 .. n_pages - 1 and every token
id taken from the prompt or from sb_seqs.root into 0 .. vocab - 1; with
debug on they also raise a bit of the context's status word, which
sb_device_check reports as SB_EDEVICE and clears.  Checked here on the tiny
fp32 model (two sequences, weights generated on the device):

* valid inputs report nothing over a whole iteration;
* a prompt with ids past the vocabulary and negative ones is reported
  ("token") and computes exactly what the prompt with those ids clamped
  computes (the roots and every K/V cache entry bit-identical);
* a root token past the vocabulary is reported at the first expansion;
* page-table entries past n_pages and negative ones are reported ("page")
  by verification (the 16-row kernel, and the 32x32 kernel at the
  16-sequence bf16 shape), and a check after the report comes back clean;
* with debug off the same inputs report nothing.

No oracle is involved: the property is the library's own.
"""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from paper_2605_07243_amd import binding as B
from paper_2605_07243_amd.runtime import Runtime

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(300)]

W = dataclasses.replace(synth.WORKLOADS["tiny-fp32"], n_seqs=2,
                        prompt_len=(40, 70))


def _prompts():
    return [list(map(int, p)) for p in synth.prompts(W)]


def _expect_report(rt, kind):
    with pytest.raises(B.SBError) as e:
        rt.device_check()
    assert e.value.code == B.SB_EDEVICE
    assert kind in str(e.value), str(e.value)
    rt.device_check()        # the report cleared the word


def test_valid_inputs_report_nothing():
    rt = Runtime(W, None, seed=11)
    rt.set_debug(True)
    rt.prefill(_prompts())
    rt.iteration()
    rt.iteration()
    rt.device_check()


def test_out_of_range_prompt_tokens_are_clamped_and_reported():
    V = W.target.vocab
    bad = _prompts()
    bad[0][3] = V + 5
    bad[0][-1] = -7
    bad[1][0] = 2 * V
    good = [[min(max(t, 0), V - 1) for t in p] for p in bad]
    rt_bad = Runtime(W, None, seed=12)
    rt_bad.set_debug(True)
    print("[debug] prefill with out-of-range prompt ids", flush=True)
    rt_bad.prefill(bad)
    _expect_report(rt_bad, "token id")
    rt_good = Runtime(W, None, seed=12)
    rt_good.set_debug(True)
    rt_good.prefill(good)
    rt_good.device_check()
    torch.cuda.synchronize()
    assert torch.equal(rt_bad.root, rt_good.root)
    assert torch.equal(rt_bad.T, rt_good.T)
    for a, b in ((rt_bad.tk, rt_good.tk), (rt_bad.tv, rt_good.tv),
                 (rt_bad.dk, rt_good.dk), (rt_bad.dv, rt_good.dv)):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_out_of_range_root_token_is_reported():
    rt = Runtime(W, None, seed=13)
    rt.set_debug(True)
    rt.prefill(_prompts())
    rt.device_check()
    rt.root[1] = W.target.vocab + 100
    rt.expand(1)
    _expect_report(rt, "token id")


def test_out_of_range_pages_are_reported():
    rt = Runtime(W, None, seed=14)
    rt.set_debug(True)
    rt.prefill(_prompts())
    for m in range(1, W.M + 1):
        rt.expand(m)
    rt.device_check()
    n_pages = rt.tpt.numel()
    saved = rt.tpt.clone()
    rt.tpt[0, 0] = n_pages + 5      # a committed prefix page of sequence 0
    rt.tpt[1, 1] = -1               # and one of sequence 1
    print("[debug] verify over out-of-range page-table entries", flush=True)
    rt.verify()
    _expect_report(rt, "page-table entry")
    rt.set_debug(False)
    rt.verify()
    rt.device_check()               # debug off: nothing is reported
    rt.tpt.copy_(saved)
    rt.set_debug(True)
    rt.verify()
    rt.device_check()


def test_out_of_range_pages_are_reported_by_the_32x32_kernel():
    """The same at the 16-sequence bf16 shape (one target layer, weights
    generated on the device), where verification runs the 32x32 kernel."""
    w = synth.with_layers(synth.WORKLOADS["llama3-8b-batch16-paged"], 1)
    rt = Runtime(w, None, seed=15)
    rt.set_debug(True)
    rt.prefill(synth.prompts(w))
    for m in range(1, w.M + 1):
        rt.expand(m)
    rt.device_check()
    saved = rt.tpt.clone()
    rt.tpt[3, 0] = rt.tpt.numel() + 1
    print("[debug] 32x32 verify over an out-of-range page-table entry",
          flush=True)
    rt.verify()
    _expect_report(rt, "page-table entry")
    rt.tpt.copy_(saved)
    rt.verify()
    rt.device_check()
