"""GPU parity on the tiny fp32 workload (2-layer target, d = 256, 4 heads,
vocab 1024, K = 4, M = 3, budget 32, prompt 128): every C-ABI call against
the oracle on identical inputs (the oracle's state is copied into the device
caches before each call), tolerance 1e-4 relative for fp32."""
import copy
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import specdec

from gpu_harness import host, inject, models, rel_err, runtime

pytestmark = pytest.mark.gpu
TOL = 1e-4


@pytest.fixture(scope="module")
def tiny():
    w = synth.WORKLOADS["tiny-fp32"]
    weights, tgt, dr = models(w)
    prompt = synth.prompts(w)[0]
    st = specdec.prefill(tgt, dr, prompt)
    rt = runtime(w, weights, max_pages=32, adapt_cap=8)
    return w, tgt, dr, prompt, st, rt


def test_prefill(tiny):
    w, tgt, dr, prompt, st, rt = tiny
    print("prefill", flush=True)
    rt.prefill([prompt])
    torch.cuda.synchronize()
    assert int(rt.T[0]) == st.T
    assert int(rt.root[0]) == st.root
    assert rel_err(host(rt.cond_taps[0]), st.cond_taps).max() < TOL
    k, v = rt.read_cache("target", 0, st.T)
    for layer in range(w.target.n_layers):
        assert rel_err(k[layer].reshape(st.T, -1),
                       st.tkv.k[layer].reshape(st.T, -1)).max() < TOL
        assert rel_err(v[layer].reshape(st.T, -1),
                       st.tkv.v[layer].reshape(st.T, -1)).max() < TOL
    k, v = rt.read_cache("drafter", 0, st.T)
    assert rel_err(k[0].reshape(st.T, -1), st.dkv.k[0].reshape(st.T, -1)).max() < TOL
    assert rel_err(v[0].reshape(st.T, -1), st.dkv.v[0].reshape(st.T, -1)).max() < TOL


def _check_block(rt, exp, rec_rows, tree_nodes, m):
    d = rt.dout
    n_call = int(d["n_call"][0])
    assert n_call == exp["R"], (n_call, exp["R"])
    call_row = host(d["call_row"])[:n_call]
    lg = host(d["logits"])[:n_call]
    base = exp["base"]
    assert list(call_row) == list(range(base, base + exp["R"]))
    assert rel_err(lg, exp["logits"]).max() < TOL
    for i in range(exp["R"]):
        r = rec_rows[base + i]
        o = base + i
        assert list(host(d["topk_id"][0, o])) == list(r.topk), (m, i)
        assert abs(float(d["lse"][0, o]) - r.lse) < TOL * max(1, abs(r.lse))
        assert rel_err(host(d["psi"][0, o]), r.psi) < TOL
        assert int(d["bucket"][0, o]) == r.bucket
        assert int(d["branch"][0, o]) == r.branch
        assert rel_err(host(rt.tree["h_last"][0, o]), r.h_last) < TOL


def test_iteration_calls(tiny):
    """Block expansions, verification, acceptance and commit, each on the
    oracle's own inputs."""
    w, tgt, dr, prompt, st0, rt = tiny
    _iteration_case(w, st0, rt)


@pytest.mark.parametrize("budget", [2, 5, 9])
def test_iteration_calls_small_budget(tiny, budget):
    """Degenerate trees: a budget of 2, 5 or 9 nodes fills during block 1
    (the last rows of the block are cut), so blocks 2 and 3 have no starts
    and must add nothing; verify, accept and commit then run on the cut
    tree (Alg. 2 with the tree budget of Sec. 3.2)."""
    w0, tgt, dr, prompt, st0, _ = tiny
    w = dataclasses.replace(w0, budget=budget)
    weights, _, _ = models(w)
    rt = runtime(w, weights, max_pages=32, adapt_cap=8)
    _iteration_case(w, st0, rt, tgt, dr)


def _iteration_case(w, st0, rt, tgt=None, dr=None):
    if tgt is None:
        weights, tgt, dr = models(w)
    st = copy.deepcopy(st0)
    inject(rt, 0, st)
    ref_state = copy.deepcopy(st)
    rec = specdec.iteration(tgt, dr, ref_state, w)
    tree = rec["tree"]
    for m, exp in enumerate(rec["expansions"], start=1):
        print("expand", m, flush=True)
        rt.expand(m, want_logits=True)
        torch.cuda.synchronize()
        _check_block(rt, exp, rec["rows"], tree, m)
    for m in range(len(rec["expansions"]) + 1, w.M + 1):
        print("expand", m, "(no starts)", flush=True)
        rt.expand(m, want_logits=True)
        torch.cuda.synchronize()
        assert int(rt.dout["n_call"][0]) == 0, m
    n = len(tree)
    assert int(rt.tree["n_nodes"][0]) == n
    t = rt.tree
    for j, nd in enumerate(tree.nodes):
        assert int(t["token"][0, j]) == nd.token, j
        assert int(t["parent"][0, j]) == nd.parent, j
        assert int(t["depth"][0, j]) == nd.depth, j
        assert int(t["rank"][0, j]) == nd.rank, j
        assert int(t["row"][0, j]) == nd.row, j
        assert abs(float(t["cum_logp"][0, j]) - nd.cum_logp) < 1e-3
    mask = tree.mask()
    anc = host(t["anc"][0]).view(np.uint32)
    for j in range(n):
        bits = [(anc[j, q >> 5] >> (q & 31)) & 1 for q in range(n)]
        assert np.array_equal(np.array(bits, bool), mask[j]), j
    print("verify", flush=True)
    rt.verify(want_logits=True)
    torch.cuda.synchronize()
    vl = host(rt.vout["logits"])[:n]
    assert rel_err(vl, rec["verify_logits"]).max() < TOL
    assert list(host(rt.vout["argmax"][0, :n])) == list(rec["greedy"])
    assert rel_err(host(rt.vout["taps"][0, :n]).reshape(n * 3, -1),
                   rec["taps"].reshape(n * 3, -1)).max() < TOL
    print("accept", flush=True)
    rt.accept()
    torch.cuda.synchronize()
    a = int(rt.aout["n_accepted"][0])
    assert a == len(rec["path"])
    assert list(host(rt.aout["path"][0, :a])) == rec["path"]
    assert int(rt.aout["bonus"][0]) == rec["bonus"]
    # verifier-derived signal at the rejected position
    rg, rr = float(rt.aout["r_reject"][0]), rec["r_reject"]
    if rr is None:
        assert rg == -1.0
    else:
        assert abs(rg - rr) <= 1e-3 * rr + 1e-9, (rg, rr)
    # the adaptation buffer takes the rejected position's row and token
    buf = rt.adapt_buffer()
    rt.adapt_push(buf)
    torch.cuda.synchronize()
    cont = specdec.continuing_row(tree, rec["rows"], (rec["path"] or [0])[-1],
                                  w.K)
    if cont is None:
        assert int(buf["count"][0]) == 0
    else:
        assert int(buf["count"][0]) == 1
        assert int(buf["target"][0]) == rec["bonus"]
        assert rel_err(host(buf["h"][0]), rec["rows"][cont].h_last) < TOL
    print("commit", flush=True)
    rt.commit()
    torch.cuda.synchronize()
    assert int(rt.T[0]) == ref_state.T
    assert int(rt.root[0]) == ref_state.root
    assert rel_err(host(rt.cond_taps[0]), ref_state.cond_taps).max() < TOL
    T0 = st.T
    k, v = rt.read_cache("target", 0, ref_state.T - T0, T0)
    for layer in range(w.target.n_layers):
        ref = ref_state.tkv.k[layer][T0:]
        assert rel_err(k[layer].reshape(len(ref), -1), ref.reshape(len(ref), -1)).max() < TOL
    k, v = rt.read_cache("drafter", 0, ref_state.T - T0, T0)
    ref = ref_state.dkv.k[0][T0:]
    assert rel_err(k[0].reshape(len(ref), -1), ref.reshape(len(ref), -1)).max() < TOL
    ref = ref_state.dkv.v[0][T0:]
    assert rel_err(v[0].reshape(len(ref), -1), ref.reshape(len(ref), -1)).max() < TOL


def test_lossless_loop(tiny):
    """Losslessness on the device: the committed stream of the HIP loop
    equals the target's greedy decode."""
    w, tgt, dr, prompt, st0, rt = tiny
    ref = specdec.greedy_decode(tgt, prompt, 24)
    rt.prefill([prompt])
    torch.cuda.synchronize()
    out = [int(rt.root[0])]
    while len(out) < 24:
        rt.iteration()
        torch.cuda.synchronize()
        a = int(rt.aout["n_accepted"][0])
        path = host(rt.aout["path"][0, :a])
        toks = host(rt.tree["token"][0])
        out += [int(toks[p]) for p in path] + [int(rt.aout["bonus"][0])]
    assert out[:24] == ref


@pytest.mark.parametrize("temperature", [1.0, 0.25])
def test_iteration_sampling(tiny, temperature):
    """One whole iteration with stochastic verification on both sides (the
    same float32 uniforms): drafting, verification logits, the walk, the
    bonus draw and the commit.  The accepted path and bonus must be equal
    where the oracle's decision margins exceed the float32 error (1e-4 for
    the acceptance tests, 2e-6 of the residual mass for the draw); the
    device state after the commit must then equal the oracle's."""
    from oracle.sampling import accept_sample
    w, tgt, dr, prompt, st0, rt = tiny
    st = copy.deepcopy(st0)
    inject(rt, 0, st)
    rng = np.random.default_rng(int(temperature * 1000))
    ua = rng.random((1, w.budget)).astype(np.float32)
    ub = rng.random((1, w.budget)).astype(np.float32)
    ref_state = copy.deepcopy(st)
    rec = specdec.iteration(tgt, dr, ref_state, w,
                            sampling=(temperature, ua[0].astype(np.float64),
                                      ub[0].astype(np.float64)))
    margins = accept_sample(rec["tree"], rec["verify_logits"], temperature,
                            ua[0].astype(np.float64), ub[0].astype(np.float64))
    assert margins["path"] == rec["path"] and margins["bonus"] == rec["bonus"]
    for m in range(1, w.M + 1):
        rt.expand(m)
    rt.verify(want_logits=True)
    rt.accept_sample(temperature, torch.as_tensor(ua).to(rt.dev),
                     torch.as_tensor(ub).to(rt.dev))
    torch.cuda.synchronize()
    n = len(rec["tree"])
    assert int(rt.tree["n_nodes"][0]) == n
    assert list(host(rt.tree["token"][0, :n])) == \
        [nd.token for nd in rec["tree"].nodes]
    if margins["test_margin"] <= 1e-4 or margins["cdf_margin"] <= 2e-6:
        pytest.skip(f"decision within float32 error (margins "
                    f"{margins['test_margin']:.2e}, {margins['cdf_margin']:.2e})")
    a = int(rt.aout["n_accepted"][0])
    assert list(host(rt.aout["path"][0, :a])) == rec["path"]
    assert int(rt.aout["bonus"][0]) == rec["bonus"]
    rt.commit()
    torch.cuda.synchronize()
    assert int(rt.T[0]) == ref_state.T
    assert int(rt.root[0]) == ref_state.root
    assert rel_err(host(rt.cond_taps[0]), ref_state.cond_taps).max() < TOL
