"""Shared set-up for the GPU parity tests: one workload, the oracle and the
HIP runtime built from the same synth weights, and helpers that copy an
oracle state into the device caches (teacher forcing: oracle -> device
only) and compare per-call outputs."""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import specdec
from oracle.model import Drafter, Target


def models(w, seed=0, jitter=0.1):
    tw = synth.make_weights(synth.target_specs(w.target), seed, w.dtype,
                            jitter=jitter)
    dw = synth.drafter_weights(w, seed, jitter=jitter)
    tgt = Target(tw, w.target, w.dtype, w.tap_layers)
    dr = Drafter(dw, w.target, w.dtype, w.drafter_layers, tgt.embed)
    return {**tw, **dw}, tgt, dr


def runtime(w, weights, **kw):
    from paper_2605_07243_amd.runtime import Runtime
    return Runtime(w, weights, **kw)


def inject(rt, seq: int, st: specdec.SeqState):
    """Copy an oracle sequence state into the device caches and state."""
    rt.write_cache("target", seq, st.tkv.k, st.tkv.v, 0)
    rt.write_cache("drafter", seq, st.dkv.k, st.dkv.v, 0)
    rt.root[seq] = int(st.root)
    rt.T[seq] = int(st.T)
    rt.cond_taps[seq] = torch.as_tensor(np.asarray(st.cond_taps, np.float32))
    rt.set_length_bound(0)
    torch.cuda.synchronize()


def rel_err(a, b):
    """max |a - b| / max |b| per row (last axis)."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return (np.abs(a - b).max(axis=-1) / np.maximum(np.abs(b).max(axis=-1),
                                                    1e-30))


def host(t):
    return t.detach().cpu().numpy()
