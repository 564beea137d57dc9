#!/usr/bin/env python
"""SpecBlock hot-path benchmark on one MI355X.

A step is one verifier iteration of the whole hot path on the
Llama-3-8B-shaped workload (random-init bf16 target, 32 layers, d 4096,
32/8 heads, MLP 14336, vocab 128256; one-layer drafter of the same shape;
K = 4, M = 2 block expansions, tree budget 60, batch 1, prompt of 1024
uniform-random ids): M sb_draft_block_expand calls, sb_tree_verify,
sb_accept and sb_commit, with inputs resident in HBM.

Prints one JSON line: value = committed (accepted + bonus) tokens per second
over the timed steps; block-expansion steps/s and tree-attention HBM GB/s
from HIP events on the library's stream; the roofline of the dominant
kernel (the projection GEMMs: HBM-bound with few rows per call, MFMA-bound
with many, decided by arithmetic intensity against the ridge point); and the
CPU oracle timed on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 MFMA, MI355X
BUCKET_SEED = 11
METRIC = ("block-expansion steps/s + tree-attn HBM GB/s; accepted tokens/s "
          "(8B-shape)")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def attn_bytes(w, T_total, n_nodes, rows_block, es):
    """Algorithmic bytes of the tree-attention launches of one iteration:
    every committed prefix K/V entry of every sequence (T_total entries over
    the batch) and every segment entry read once per layer, Q read and O
    written once per row."""
    s = w.target
    kv_entry = 2 * s.n_kv_heads * s.head_dim * es
    q_row = s.n_heads * s.head_dim * es * 2
    verify = s.n_layers * (T_total * kv_entry + n_nodes * kv_entry
                           + n_nodes * q_row)
    draft = 0.0
    for rows in rows_block:
        draft += w.drafter_layers * (T_total * kv_entry + rows * kv_entry
                                     + rows * q_row)
    return verify + draft


def attn_flops(w, verify_nodes_T, draft_rows_T):
    """Algorithmic flops of the tree-attention launches (2 per multiply-add:
    the scores and the probability-weighted sum of the values) over the
    committed prefix: every verified node and every drafter row attends to
    the T entries of its sequence in every layer (the sums over nodes and
    rows of T are the arguments); the at most M K + 1 tree keys per row are
    left out."""
    s = w.target
    per = 4.0 * s.n_heads * s.head_dim
    return per * (s.n_layers * verify_nodes_T + w.drafter_layers * draft_rows_T)


def gemm_flops(w, verify_rows, rows_block, n_seqs):
    """Algorithmic flops (2 per multiply-add) of the projection GEMMs over
    the actual rows: verify rows through every target layer and the LM
    head; each block's drafter rows through W_fuse, the drafter layers (with
    the shift) and the LM head; block 1 also the condition projection."""
    s = w.target
    d, F = s.d_model, s.d_ff
    layer = (s.n_heads + 2 * s.n_kv_heads) * s.head_dim * d \
        + d * s.n_heads * s.head_dim + 2 * F * d + d * F
    lm = s.vocab * d
    lm_d = (w.draft_vocab or s.vocab) * d
    fl = 2.0 * verify_rows * (s.n_layers * layer + lm)
    for i, rows in enumerate(rows_block):
        fl += 2.0 * rows * (3 * d * d + w.drafter_layers * (layer + 2 * d * d)
                            + lm_d)
        if i % w.M == 0:
            fl += 2.0 * n_seqs * 3 * d * d
    return fl


def gemm_traffic(workload):
    """Measured HBM bytes per projection-GEMM dispatch from the committed
    counter summary of this workload, or None when there is none or the
    GEMM sources changed since it was taken."""
    from paper_2605_07243_amd.profile_summary import gemm_sources_sha256
    path = os.path.join(ROOT, "profiles", f"gemm_traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("sources_sha256") != gemm_sources_sha256():
        log("gemm traffic summary is stale (sources changed); traffic = null")
        return None
    return d["bytes_per_dispatch"]


def cpu_baseline(w, T, budget_s=10.0, buckets="natural"):
    """Time the CPU oracle on a bounded sample of the workload: whole
    iterations of the real shapes (M block expansions of the drafter over a
    prefix of T entries, then the verify forward of the drafted tree through
    n_layers decoder layers and the LM head), repeated until budget_s of CPU
    time has passed.  To bound memory, the verify layers all use the weights
    and prefix cache of one generated layer: the arithmetic per layer is that
    of a real layer.  buckets: "paper" / "uniform" force the drafter rows'
    buckets as the GPU run does (seeded paper-frequency draws / all b1)."""
    import dataclasses

    import numpy as np
    from threadpoolctl import threadpool_info

    import synth
    from oracle import specdec
    from oracle.model import Drafter, Target, decoder_layer
    from oracle.numerics import rmsnorm

    w1 = synth.with_layers(w, 1)
    w1 = dataclasses.replace(w1, target=dataclasses.replace(w1.target),
                             prompt_len=(T, T))
    t0 = time.perf_counter()
    tw = synth.target_weights(w1, seed=0)
    dw = synth.drafter_weights(w1, seed=0)
    tgt = Target(tw, w1.target, w1.dtype, (0, 0, 0))
    dr = Drafter(dw, w1.target, w1.dtype, w1.drafter_layers, tgt.embed)
    del tw, dw
    log(f"cpu baseline: weights ready in {time.perf_counter() - t0:.1f}s")
    s = w1.target
    rng = np.random.default_rng(7)
    st = specdec.SeqState([], T, int(rng.integers(s.vocab)),
                          tgt.new_prefix(), dr.new_prefix(),
                          rng.standard_normal((3, s.d_model)))
    k, v = synth.random_kv(1, "bench.t", T, s, w1.dtype)
    st.tkv.k[0], st.tkv.v[0] = k.astype(np.float64), v.astype(np.float64)
    k, v = synth.random_kv(1, "bench.d", T, s, w1.dtype)
    st.dkv.k[0], st.dkv.v[0] = k.astype(np.float64), v.astype(np.float64)

    def iteration(i):
        forced = None
        if buckets == "paper":
            forced = synth.paper_buckets(BUCKET_SEED, i, 1, w1.rows_per_seq)[0]
        elif buckets == "uniform":
            forced = synth.uniform_buckets(1, w1.rows_per_seq)[0]
        tree = specdec.DraftTree(st.root, w1.budget)
        rows = []
        seg = dr.new_segment(w1.rows_per_seq)
        starts = [specdec.Start(0, st.root, st.T,
                                dr.cond_from_taps(st.cond_taps), [])]
        t = time.perf_counter()
        for m in range(1, w1.M + 1):
            if not starts:
                break
            rec = specdec.expand_block(dr, st, tree, rows, seg, starts, w1.K,
                                       m, w1.branch_map, forced)
            if m < w1.M:
                picks = specdec.select_starts(tree, rows, rec["alive"],
                                              rec["chain"], rec["first_new"],
                                              w1.B_max)
                starts = [specdec.start_from_node(tree, rows, st, n)
                          for n in picks]
        t_draft = time.perf_counter() - t
        n = len(tree)
        tseg = tgt.new_segment(n)
        x = tgt.embed[[nd.token for nd in tree.nodes]]
        pos = np.array([st.T + nd.depth for nd in tree.nodes])
        vis = [tree.anc_or_self(i) for i in range(n)]
        for _ in range(w.target.n_layers):
            x = decoder_layer(tgt.layers[0], x, pos, np.arange(n), vis,
                              st.tkv.k[0], st.tkv.v[0], tseg.k[0], tseg.v[0],
                              s, tgt.num)
        z = tgt.num.act(rmsnorm(x, tgt.final_norm, s.norm_eps)) @ tgt.lm_head.T
        _ = [specdec.argmax_low(r) for r in z]
        return t_draft, len(rows), n

    t_start = time.perf_counter()
    iters, t_draft, rows, n = 0, 0.0, 0, 0
    while True:
        td, rows, n = iteration(iters)
        t_draft += td
        iters += 1
        elapsed = time.perf_counter() - t_start
        if elapsed >= budget_s:
            break
    blas = [i.get("num_threads") for i in threadpool_info()
            if i.get("user_api") == "blas"]
    cores = int(max(blas)) if blas else 1
    return {
        "value": round(iters / elapsed, 4),
        "unit": "tokens/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"float64 oracle, {iters} whole iteration(s) in "
                   f"{elapsed:.1f}s: {w1.M} block expansions ({rows} drafter "
                   f"rows, prefix {T}) + verify of {n} nodes through "
                   f"{w.target.n_layers} decoder layers (weights of one "
                   f"generated layer) + LM head; 1 committed token per "
                   f"iteration (random weights)"),
        "block_expansion_steps_per_s": round(iters * w1.M / t_draft, 4),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama3-8b-k4")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--buckets", choices=("natural", "paper", "uniform"),
                    default="natural",
                    help="natural: the rank head's argmax decides each "
                         "drafter row's bucket; paper: buckets are forced "
                         "from seeded draws with the class frequencies of "
                         "a trained drafter (b0..b3 = 75.2/15.0/4.1/5.7%%), "
                         "which shapes the trees like the paper's; uniform: "
                         "the fixed-k tree of the rank-guided-branching "
                         "ablation (every row b1, every bucket branches "
                         "--uniform-k)")
    ap.add_argument("--uniform-k", type=int, default=3)
    ap.add_argument("--temperature", type=float, default=0.0,
                    help="0: greedy acceptance; > 0: stochastic tree "
                         "verification at this temperature (the paper's "
                         "sampling setting is 1.0), with seeded uniforms "
                         "resident on the device")
    ap.add_argument("--e2e-tokens", type=int, default=256,
                    help="after the timed steps, decode until every sequence "
                         "has this many new tokens and report the wall time "
                         "of that loop (host loop and per-iteration "
                         "synchronisation included); 0 skips it")
    ap.add_argument("--calib-mib", type=int, default=0,
                    help="before warmup, run a plain elementwise copy "
                         "(torch.neg) of this many MiB three times, to "
                         "calibrate HBM byte counters against a kernel of "
                         "known traffic")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (got --gpus "
              f"{args.gpus}); the multi-GPU sharding plan is design-only",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2605_07243_amd.runtime import Runtime

    w = synth.WORKLOADS[args.workload]
    if args.buckets == "uniform":
        w = synth.uniform_tree(w, args.uniform_k)
    es = 2 if w.dtype == "bf16" else 4
    log(f"workload {w.name}: allocating and generating weights on device")
    t = time.perf_counter()
    rt = Runtime(w, None, seed=0)
    torch.cuda.synchronize()
    log(f"weights + buffers in {time.perf_counter() - t:.1f}s")
    prompts = synth.prompts(w)
    t = time.perf_counter()
    rt.prefill(prompts)
    torch.cuda.synchronize()
    log(f"prefill {sum(len(p) for p in prompts)} tokens in "
        f"{time.perf_counter() - t:.2f}s")
    # forced buckets: one [n_seqs][row_cap] draw per iteration (warmup, timed
    # pass, profiled pass), resident on the device before timing
    sched = None
    n_iter = args.warmup + 2 * args.steps
    if args.buckets == "paper":
        import numpy as np
        sched = torch.as_tensor(np.stack(
            [synth.paper_buckets(BUCKET_SEED, i, rt.S, rt.row_cap)
             for i in range(n_iter)])).to(rt.dev)
    elif args.buckets == "uniform":
        sched = torch.as_tensor(synth.uniform_buckets(
            rt.S, rt.row_cap)).to(rt.dev).expand(n_iter, -1, -1)
    it = [0]

    def next_iteration():
        if sched is not None:
            rt.set_buckets(sched[it[0]])
        it[0] += 1

    sampling = args.temperature > 0
    if sampling:
        g = torch.Generator(device=rt.dev)
        g.manual_seed(13)
        u_acc = torch.rand((n_iter, rt.S, w.budget), generator=g,
                           device=rt.dev)
        u_bon = torch.rand((n_iter, rt.S, w.budget), generator=g,
                           device=rt.dev)

    def verify_accept():
        """Verification and acceptance of the iteration just drafted."""
        if sampling:
            rt.verify(want_logits=True)
            i = it[0] - 1
            rt.accept_sample(args.temperature, u_acc[i], u_bon[i])
        else:
            rt.verify()
            rt.accept()

    if args.calib_mib:
        src = torch.ones(args.calib_mib << 18, device=rt.dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
    for i in range(args.warmup):
        next_iteration()
        for m in range(1, w.M + 1):
            rt.expand(m)
        verify_accept()
        rt.commit()
    torch.cuda.synchronize()
    log("warmup done")

    stream = torch.cuda.current_stream()
    # events: before block 1, after each block m, after verify/accept/commit
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(w.M + 2)]
          for _ in range(args.steps)]
    T0 = rt.T.clone()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        next_iteration()
        ev[i][0].record(stream)
        for m in range(1, w.M + 1):
            rt.expand(m)
            ev[i][m].record(stream)
        verify_accept()
        rt.commit()
        ev[i][w.M + 1].record(stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    committed = int((rt.T - T0).sum())
    block1_ms = sum(e[0].elapsed_time(e[1]) for e in ev)
    later_ms = sum(e[1].elapsed_time(e[w.M]) for e in ev)
    draft_ms = block1_ms + later_ms
    rest_ms = sum(e[w.M].elapsed_time(e[w.M + 1]) for e in ev)

    def median(xs):
        xs = sorted(xs)
        h = len(xs) // 2
        return xs[h] if len(xs) % 2 else 0.5 * (xs[h - 1] + xs[h])

    med_step = median([e[0].elapsed_time(e[w.M + 1]) for e in ev])
    med_block1 = median([e[0].elapsed_time(e[1]) for e in ev])
    med_later = (median([e[1].elapsed_time(e[w.M]) / (w.M - 1) for e in ev])
                 if w.M > 1 else None)
    log(f"timed {args.steps} steps in {dt:.3f}s: {committed} tokens, "
        f"draft {draft_ms / args.steps:.3f} ms/step (block 1 "
        f"{block1_ms / args.steps:.3f}), verify+accept+commit "
        f"{rest_ms / args.steps:.3f} ms/step")

    # second pass over the same work with per-kernel HIP events
    Tp0 = rt.T.clone()
    rows_block = []
    verify_rows = 0
    verify_nodes_T = draft_rows_T = 0.0   # sums of the rows' prefix lengths
    rt.profile(True)
    for i in range(args.steps):
        next_iteration()
        Ts = rt.T.cpu().numpy().astype(np.float64)
        for m in range(1, w.M + 1):
            rt.expand(m)
            n_call = int(rt.dout["n_call"][0])
            rows_block.append(n_call)
            cs = rt.dout["call_seq"][:n_call].cpu().numpy()
            draft_rows_T += float(Ts[cs].sum())
        nodes = rt.tree["n_nodes"].cpu().numpy()
        verify_rows += int(nodes.sum())
        verify_nodes_T += float((nodes * Ts).sum())
        verify_accept()
        rt.commit()
    torch.cuda.synchronize()
    rt.profile(False)
    prof = rt.profile_read()
    Tp1 = rt.T.clone()
    T_total = float((Tp0.sum() + Tp1.sum()) / 2)
    n_nodes = int(rt.tree["n_nodes"].sum())
    gemm = prof["gemm"]
    gemm_gbps = gemm["bytes"] / (gemm["ms"] * 1e-3) / 1e9
    # bytes and flops over the rows each launch processed (the library
    # captures every profiled launch's live row count); the host-side count
    # of the same flops must agree
    flops = gemm["flops"]
    flops_host = gemm_flops(w, verify_rows, rows_block, rt.S)
    if abs(flops - flops_host) > 1e-6 * flops_host:
        log(f"note: library flops {flops:.4e} vs host count {flops_host:.4e} "
            "(catch-up rows or rows past the budget)")
    gemm_tflops = flops / (gemm["ms"] * 1e-3) / 1e12
    groups = {}
    for name, g in prof["gemm_groups"].items():
        if g["launches"] == 0:
            continue
        sec = g["ms"] * 1e-3
        gb = (g["bytes_read"] + g["bytes_written"]) / sec / 1e9
        groups[name] = {
            "launches_per_step": round(g["launches"] / args.steps, 2),
            "launches_with_rows_per_step": round(
                g["launches_with_rows"] / args.steps, 2),
            "us_per_step": round(g["ms"] * 1e3 / args.steps, 1),
            "read_bytes_per_step": round(g["bytes_read"] / args.steps),
            "write_bytes_per_step": round(g["bytes_written"] / args.steps),
            "hbm_gbps": round(gb, 1), "hbm_frac": round(gb / HBM_PEAK_GBPS, 4),
            "mfma_tflops": round(g["flops"] / sec / 1e12, 1),
            "mfma_frac": round(g["flops"] / sec / 1e12 /
                               MFMA_BF16_PEAK_TFLOPS, 4)}
    # bound by arithmetic intensity against the ridge point of the chip
    ridge = MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBPS * 1e9)
    mfma_bound = flops / gemm["bytes"] > ridge
    ab = sum(attn_bytes(w, T_total, n_nodes, rows_block[i * w.M:(i + 1) * w.M],
                        es) for i in range(args.steps))
    attn = prof["tree_attn"]
    attn_gbps = ab / (attn["ms"] * 1e-3) / 1e9
    af = attn_flops(w, verify_nodes_T, draft_rows_T)
    attn_tflops = af / (attn["ms"] * 1e-3) / 1e12
    log(f"gemm {gemm['launches']} launches {gemm['ms']:.2f} ms "
        f"{gemm_gbps:.0f} GB/s {gemm_tflops:.0f} TFLOP/s; tree-attn {attn['launches']} launches "
        f"{attn['ms']:.2f} ms {attn_gbps:.0f} GB/s; vocab "
        f"{prof['vocab']['ms']:.2f} ms")

    traffic = gemm_traffic(w.name)
    if traffic is not None:
        traffic = round(traffic)
    out = {
        "metric": METRIC,
        "value": round(committed / dt, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dt * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic: random-init N(0,0.02) weights, uniform random "
                "prompt ids",
        "config": {"workload": w.name,
                   "target": (f"Llama-3-shaped, {w.target.n_layers} layers, "
                              f"d {w.target.d_model}"),
                   "drafter_layers": w.drafter_layers,
                   "draft_vocab": w.draft_vocab or w.target.vocab,
                   "n_seqs": w.n_seqs, "prompt_len": list(w.prompt_len),
                   "K": w.K, "M": w.M, "B_max": w.B_max,
                   "budget": w.budget, "branch_map": list(w.branch_map),
                   "buckets": {
                       "natural": "natural (random rank head)",
                       "paper": "paper-frequency (forced, seeded draws "
                                "75.2/15.0/4.1/5.7%)",
                       "uniform": f"uniform fixed-{args.uniform_k} tree "
                                  "(forced b1)"}[args.buckets],
                   "decoding": (f"sampling T={args.temperature:g}"
                                if sampling else "greedy")},
        "block_expansion_steps_per_s": round(w.M * args.steps /
                                             (draft_ms * 1e-3), 2),
        "block1_steps_per_s": round(args.steps / (block1_ms * 1e-3), 2),
        "later_block_steps_per_s": (round((w.M - 1) * args.steps /
                                          (later_ms * 1e-3), 2)
                                    if w.M > 1 else None),
        "median_ms_per_step": round(med_step, 4),
        "median_block1_ms": round(med_block1, 4),
        "median_later_block_ms": (round(med_later, 4) if med_later is not None
                                  else None),
        "verify_nodes_per_step": round(verify_rows / args.steps, 2),
        "drafter_rows_per_step": round(sum(rows_block) / args.steps, 2),
        "tree_attn_gbps": round(attn_gbps, 1),
        "tree_attn_frac": round(attn_gbps / HBM_PEAK_GBPS, 4),
        # the same launches against the MFMA peak (the bound where the
        # arithmetic intensity, rows x query heads per KV head, passes the
        # ridge: one sequence of 128 nodes, the 70B shape)
        "tree_attn_tflops": round(attn_tflops, 1),
        "tree_attn_mfma_frac": round(attn_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "tree_attn_flop_per_byte": round(af / ab, 1),
        "accepted_tokens_per_s": round(committed / dt, 3),
        "tau": round(committed / (args.steps * rt.S), 3),
        # labelled projection, not a measurement: the same iteration rate
        # with the paper's mean accepted length (Llama-3.1-8B, T = 0)
        "projected_tokens_per_s_at_paper_tau_4.41": round(
            args.steps * rt.S * 4.41 / dt, 1),
        "roofline": {"kernel": "gemm_tile_kernel (all projection GEMMs)",
                     "bound": "mfma" if mfma_bound else "hbm",
                     "achieved": round(gemm_tflops if mfma_bound
                                       else gemm_gbps, 1),
                     "peak": (MFMA_BF16_PEAK_TFLOPS if mfma_bound
                              else HBM_PEAK_GBPS),
                     "unit": "TFLOP/s" if mfma_bound else "GB/s",
                     "frac": round(gemm_tflops / MFMA_BF16_PEAK_TFLOPS
                                   if mfma_bound
                                   else gemm_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": traffic,
                     "algorithmic_bytes_per_launch": round(
                         gemm["bytes"] / max(gemm["launches"], 1)),
                     "algorithmic_read_bytes_per_step": round(sum(
                         g["bytes_read"] for g in prof["gemm_groups"].values())
                         / args.steps),
                     "algorithmic_write_bytes_per_step": round(sum(
                         g["bytes_written"]
                         for g in prof["gemm_groups"].values()) / args.steps),
                     "groups": groups,
                     "algorithmic_flops_per_launch": round(
                         flops / max(gemm["launches"], 1)),
                     "hbm_gbps": round(gemm_gbps, 1),
                     "mfma_tflops": round(gemm_tflops, 1),
                     "launches_per_step": gemm["launches"] // args.steps,
                     "avg_launch_us": round(gemm["ms"] * 1e3 /
                                            max(gemm["launches"], 1), 2)},
    }
    if args.e2e_tokens > 0:
        # end-to-end decode: iterations until every sequence has committed
        # e2e_tokens more entries, the host reading T after each iteration
        # (a serving loop's own check), within the page-table capacity
        cap_T = rt.max_pages * 16 - (w.M * w.K + 1)
        T_start = rt.T.clone().cpu()
        iters, stop = 0, False
        if sched is not None or sampling:
            e2e_mode = "greedy acceptance, rank-head buckets"
            rt.set_buckets(None)
        else:
            e2e_mode = "as the timed steps"
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        while not stop:
            for m in range(1, w.M + 1):
                rt.expand(m)
            rt.verify()
            rt.accept()
            rt.commit()
            iters += 1
            Tn = rt.T.cpu()
            stop = bool(((Tn - T_start) >= args.e2e_tokens).all()) or \
                bool((Tn > cap_T).any())
        dt_e2e = time.perf_counter() - t0
        new = int((Tn - T_start).sum())
        out["e2e"] = {"new_tokens_per_seq": int((Tn - T_start).min()),
                      "iterations": iters, "wall_s": round(dt_e2e, 4),
                      "tokens_per_s": round(new / dt_e2e, 3),
                      "decoding": e2e_mode}
        log(f"e2e: {new} tokens in {iters} iterations, {dt_e2e:.3f}s")
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        try:
            out["cpu_baseline"] = cpu_baseline(
                w, max(w.prompt_len), buckets=args.buckets)
        except MemoryError as e:
            out["cpu_baseline"] = {"error": f"oracle sample did not fit: {e}"}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
