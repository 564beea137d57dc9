"""GPU parity of the head-only drafter update (sb_head_update) against the
oracle's step, on the same buffered positions, training and pre-deployment
heads: the tiny fp32 workload (full vocabulary, row-major head) and the
paper's drafter shape on the 8B target (bf16, fragment-packed head, 32000-
token reduced vocabulary with targets inside and outside it).

Inputs come from seeded generators on the host: hidden states, targets, a
perturbed training copy of the LM head (so that the KL term is active).
The updated rank head must match within float32 error of the step; the
updated bf16 LM head must equal the oracle's step rounded to bf16, up to
one unit in the last place where the two sides' float32 / float64 sums
straddle a rounding boundary; the loss and the emptied buffer are checked.
"""
import ctypes as C
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle.adapt import head_update, logit_grads, prepare
from oracle.numerics import Numerics

from gpu_harness import host, models, runtime
from paper_2605_07243_amd import binding as B

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]


def unpack(packed: np.ndarray, rows: int, cols: int) -> np.ndarray:
    """Inverse of the fragment-packed bf16 layout (header definition)."""
    idx = np.arange(rows * cols)
    e = idx % 8
    lane = (idx // 8) % 64
    i = (idx // 512) % 4
    blk = idx // 2048
    kb, rb = blk // (rows // 32), blk % (rows // 32)
    row = 32 * rb + lane % 32
    col = 64 * kb + 32 * (lane // 32) + 8 * i + e
    out = np.empty((rows, cols), packed.dtype)
    out[row, col] = packed.reshape(-1)
    return out


CASES = {
    "tiny-fp32": ("tiny-fp32", 0, 8, 6, 0.2),
    "8b-paper-drafter": ("llama3-8b-paper-drafter", 32000, 16, 13, 0.05),
}


@pytest.mark.parametrize("name", list(CASES))
def test_head_update_matches_oracle(name):
    wname, vd, cap, n, lr = CASES[name]
    w = synth.with_layers(synth.WORKLOADS[wname], 1)
    if vd:
        w = dataclasses.replace(w, draft_vocab=vd)
    s = w.target
    d, V = s.d_model, s.vocab
    Vd = vd or V
    bf16 = w.dtype == "bf16"
    print(f"[{name}] weights", flush=True)
    weights, tgt, dr = models(w)
    rt = runtime(w, weights, adapt_cap=cap)
    rng = np.random.default_rng([21, cap])
    h = rng.standard_normal((n, d)).astype(np.float32)
    if vd:
        inside = rng.choice(dr.d2t, size=n - 3)
        outside = np.setdiff1d(np.arange(V), dr.d2t)[rng.integers(0, V - vd, 3)]
        targets = np.concatenate([inside, outside]).astype(np.int32)
    else:
        targets = rng.integers(0, V, size=n).astype(np.int32)
    buf = rt.adapt_buffer()
    buf["h"][:n] = torch.as_tensor(h)
    buf["target"][:n] = torch.as_tensor(targets)
    buf["count"][0] = n
    # training copy: the pre-deployment head plus seeded noise
    # (bf16 weights are float32 arrays of bf16-representable values)
    w0f = np.asarray(weights["d.lm_head"], np.float32)
    noise = rng.standard_normal(w0f.shape).astype(np.float32) * 0.01
    if bf16:
        wt_bits = synth.f32_to_bf16_bits(w0f + noise)
        wtf = synth.bf16_bits_to_f32(wt_bits)
    else:
        wtf = w0f + noise
    train = rt.head_copy()
    lm0 = rt._keep[4]["lm_head"]
    if bf16:
        src = torch.as_tensor(wtf).to(rt.dev).to(torch.bfloat16)  # exact
        out = torch.empty_like(src)
        assert rt.lib.sb_pack_weight(C.c_void_p(src.data_ptr()),
                                     C.c_void_p(out.data_ptr()), Vd, d,
                                     B.SB_BF16, 0, None) == B.SB_OK
        train["lm_head"].copy_(out)
    else:
        train["lm_head"].copy_(torch.as_tensor(wtf))
    rw0 = host(train["rank_w"]).astype(np.float64)
    rb0 = host(train["rank_b"]).astype(np.float64)
    loss = torch.zeros(1, dtype=torch.float32, device=rt.dev)
    kl = 0.5
    torch.cuda.synchronize()
    print(f"[{name}] update", flush=True)
    rt.head_update(buf, lm0, train, lr, kl, loss)
    torch.cuda.synchronize()
    assert int(buf["count"][0]) == 0
    # oracle step on the same values
    g = np.asarray(weights["d.final_norm"], np.float64)
    nl, nr, nb, ref_loss = head_update(
        wtf.astype(np.float64), rw0, rb0, w0f.astype(np.float64),
        h.astype(np.float64), targets, g, s.norm_eps,
        Numerics("bf16" if bf16 else "f32"), lr, kl, dr.d2t)
    got_loss = float(loss[0])
    assert abs(got_loss - ref_loss) <= 2e-3 * abs(ref_loss) + 1e-5, \
        (got_loss, ref_loss)
    for got, ref, old in ((host(train["rank_w"]), nr, rw0),
                          (host(train["rank_b"]), nb, rb0)):
        dg, dref = got.astype(np.float64) - old, ref - old
        assert np.abs(dg - dref).max() <= 2e-2 * np.abs(dref).max() + 1e-7
    if bf16:
        got = host(train["lm_head"].view(torch.int16)).view(np.uint16)
        got = synth.bf16_bits_to_f32(unpack(got, Vd, d)).astype(np.float64)
        want = synth.bf16_bits_to_f32(
            synth.f32_to_bf16_bits(nl.astype(np.float32))).astype(np.float64)
        # the applied update lr sum_i G_iv a_ik must agree within 1% of its
        # terms' magnitude lr sum_i |G_iv| max_i |a_ik| (a bf16 operand a_ik
        # rounded the other way moves a term by 0.4%) plus the storage
        # rounding (one bf16 unit of the result)
        A, ids, _, _ = prepare(wtf, h, targets, g, s.norm_eps,
                               Numerics("bf16"), dr.d2t)
        G = logit_grads(wtf, w0f, A, ids, kl)
        scale = lr * np.abs(G).sum(axis=0)[:, None] * \
            np.abs(A).max(axis=0)[None, :]
        ulp = np.maximum(np.abs(want), 1e-30) * 2.0 ** -7
        err = np.abs(got - want)
        bound = 1e-2 * scale + ulp
        moved = int((want != wtf).sum())
        exact = float((got == want).mean())
        print(f"[{name}] bf16 head: {moved} elements moved, exact "
              f"{exact:.6f}, worst err/bound {(err / bound).max():.3f}",
              flush=True)
        if not (err <= bound).all():
            bad = np.argwhere(err > bound)
            print(f"[{name}] {len(bad)} elements out of bound; rows "
                  f"{np.unique(bad[:, 0])[:20]}", flush=True)
            for r, c in bad[np.argsort(-(err / bound)[err > bound])][:8]:
                print(f"  ({r},{c}) got {got[r, c]:.6g} want {want[r, c]:.6g} "
                      f"old {wtf[r, c]:.6g} ref step {nl[r, c] - wtf[r, c]:.3g} "
                      f"bound {bound[r, c]:.3g}", flush=True)
        assert (err <= bound).all()
        assert moved > 0 and exact > 0.99
    else:
        gotw = host(train["lm_head"]).astype(np.float64)
        dg, dref = gotw - wtf, nl - wtf
        assert np.abs(dg - dref).max() <= 1e-3 * np.abs(dref).max() + 1e-9
