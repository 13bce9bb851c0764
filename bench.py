#!/usr/bin/env python3
"""Speculative-decoding step of the sparse-drafter / full-verifier path on one MI355X.

Workload (16K collapse regime): 8 sequences x 16,384 cached tokens, 32 query
heads, 8 KV heads, head_dim 128, bf16 caches; drafter budget B = 1024 (the
selection runs once, outside the timed step, as after prefill); draft length
gamma = 5; vocab 128,256.  A step is one pass of Alg. 2's per-round work:

    gamma x bd_sparse_decode_attn   (drafter cache, B selected entries)
    1     x bd_verify_attn          (verifier cache, gamma+1 rows, full KV)
    1     x bd_accept_len           (fp32 logits [8][6][128256])

The drafter and the verifier have separate caches of the same shape.  The step
is captured once in a HIP graph and replayed; inputs stay resident in HBM.
Prints one JSON line.

Besides the step time the line carries each kernel's time warm (back-to-back
launches over the same inputs, in a graph) and cold (each launch after a 512 MiB
streaming read, so the 256 MB MALL holds none of its inputs), the step's p10/median/p90
over single replays, the step at B = 512, and whether decode and verify meet
60% of the 8 TB/s HBM peak.

`--op select`, `--op multiview`, `--op multiview_bwd`, `--op paged`, `--op
updates` and `--op ce` time the other operations on their own workloads
(selection at the same 16K batch; the multi-view block at 4 x 8,192, C = 64,
four budgets, or with `--mv-workload train-c256-16k` the training shape
16,384 tokens, C = 256; the ragged paged batch of 64 MHA sequences), each as
one JSON line of the same form.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "draft+verify attention µs/step and HBM GB/s at 16K ctx, B=1024, γ=5"
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--budget", type=int, default=1024)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--op", choices=("step", "select", "multiview", "multiview_bwd", "paged", "updates", "ce"),
                    default="step")
    ap.add_argument("--mv-workload", choices=("multiview-train-b4-8k", "train-c256-16k"), default="multiview-train-b4-8k",
                    help="--op multiview / multiview_bwd: the multi-view block (4 x 8K, C = 64, token-level views) or "
                         "the training shape (1 x 16K, C = 256, TopKChunks views of every training budget)")
    ap.add_argument("--chunk", type=int, default=0,
                    help="--op select: 0 = token-level selection with pooling, s > 0 = TopKChunks with chunks of s")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only copy 512 MiB device-to-device five times (counter calibration: known bytes)")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_bytes(S, Hq, Hkv, L, B, gamma, V, D=128):
    """Bytes each call must move at least once (K/V once per KV head, q, idx, outputs, logits)."""
    dec = S * Hkv * B * D * 2 * 2 + S * Hkv * B * 4 + 2 * S * Hq * D * 2
    ver = S * Hkv * L * D * 2 * 2 + 2 * S * (gamma + 1) * Hq * D * 2
    acc = S * (gamma + 1) * V * 4 + S * gamma * 4
    return dec, ver, acc


def traffic_from_profile(kernel_src_hash: str):
    """HBM bytes per verify launch from the committed rocprofv3 counter summary, if it was
    taken on the current kernel source; otherwise None."""
    path = os.path.join(ROOT, "profiles", "verify_attn_16k_b8_counters.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("attn_source_sha256") != kernel_src_hash:
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(host, S, Hq, L, B, gamma):
    """The fp64 oracle, as it stands, on one full step of the same workload (host cores)."""
    import numpy as np

    import oracle as O
    import synth

    threads = len(os.sched_getaffinity(0))
    qs, kS, vS, kL, vL, logits, draft = host
    lens = [L] * S
    cfg = synth.workload("16k-collapse-b8")
    idx = np.stack([np.stack([np.r_[synth.random_index_set(cfg.config_id, s, g, L - cfg.window, B - cfg.window),
                                    np.arange(L - cfg.window, L)] for g in range(cfg.num_kv_heads)])
                    for s in range(S)]).astype(np.int32)
    t0 = time.perf_counter()
    for i in range(gamma):
        O.sparse_decode_attn(kS, vS, qs[:, -(gamma + 1) + i], idx, [B] * S, lens)
    O.verify_attn(kL, vL, qs[:, -(gamma + 1):], lens, gamma)
    O.accept_len(logits, draft, gamma)
    dt = time.perf_counter() - t0
    return {"value": round(dt * 1e6, 1), "unit": "us/step", "cores": threads, "kind": "oracle",
            "sample": f"one full step (5 sparse decodes B={B}, verify, accept) on all {S} sequences, fp64 numpy"}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the path needs no collectives (sequences and KV heads are "
              "independent); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2606_00144_amd as bd
    import synth

    torch.cuda.init()
    dev = torch.device("cuda:0")
    if args.copy_probe:
        x = torch.ones((128 * 1024 * 1024,), dtype=torch.float32, device=dev)   # 512 MiB
        y = torch.empty_like(x)
        for _ in range(5):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": x.numel() * 4, "copies": 5}), flush=True)
        return
    if args.op == "select":
        return bench_select(args, bd, synth, torch, np, dev)
    if args.op == "multiview":
        return bench_multiview(args, bd, synth, torch, np, dev)
    if args.op == "multiview_bwd":
        return bench_multiview_bwd(args, bd, synth, torch, np, dev)
    if args.op == "updates":
        return bench_updates(args, bd, synth, torch, np, dev)
    if args.op == "paged":
        return bench_paged(args, bd, synth, torch, np, dev)
    if args.op == "ce":
        return bench_ce(args, bd, synth, torch, np, dev)
    cfg = synth.workload("16k-collapse-b8")
    S, Hq, Hkv, L, W, gamma, V = (cfg.num_seqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.seq_len, cfg.window,
                                  cfg.gamma, cfg.vocab)
    B = args.budget

    log("generating inputs")
    qs, kS, vS = synth.kv_batch(cfg)
    _, kL, vL = synth.kv_batch(cfg, tag_k=synth.TAG_K_VERIFIER, tag_v=synth.TAG_V_VERIFIER)
    lg = [synth.logits_and_drafts(cfg, s) for s in range(S)]
    host = (np.stack(qs), np.stack(kS), np.stack(vS), np.stack(kL), np.stack(vL),
            np.stack([x[0] for x in lg]), np.stack([x[1] for x in lg]))

    def bf(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)

    q_all = bf(host[0])                                           # [S][T][Hq][D]
    kS_d, vS_d, kL_d, vL_d = bf(host[1]), bf(host[2]), bf(host[3]), bf(host[4])
    logits = torch.from_numpy(host[5]).to(dev)
    draft = torch.from_numpy(host[6]).to(dev)
    lens = torch.full((S,), L, dtype=torch.int32, device=dev)
    T = q_all.shape[1]
    q_dec = [q_all[:, T - gamma - 1 + i].contiguous() for i in range(gamma)]
    q_ver = q_all[:, T - gamma - 1:].contiguous()
    q_win = q_all[:, T - W:].contiguous()

    log("selecting the drafter's sparse cache (once, as after prefill)")
    idx, nsel = bd.bd_select_kv(kS_d, q_win, lens, B)
    B2 = 512 if B != 512 else 1024                                # the other budget of the workload
    idx2, nsel2 = bd.bd_select_kv(kS_d, q_win, lens, B2)
    torch.cuda.synchronize()

    out_dec = torch.empty((gamma, S, Hq, 128), dtype=torch.bfloat16, device=dev)
    out_ver = torch.empty_like(q_ver)
    acc = torch.empty((S,), dtype=torch.int32, device=dev)
    bonus = torch.empty((S,), dtype=torch.int32, device=dev)
    ws_dec, ws_ver, ws_acc = bd.Workspace(), bd.Workspace(), bd.Workspace()

    def decode(i, sel=None):
        ii, nn = (idx, nsel) if sel is None else sel
        bd.bd_sparse_decode_attn(kS_d, vS_d, q_dec[i], ii, nn, lens, out=out_dec[i], workspace=ws_dec)

    def verify():
        bd.bd_verify_attn(kL_d, vL_d, q_ver, lens, out=out_ver, workspace=ws_ver)

    def accept():
        bd.bd_accept_len(logits, draft, workspace=ws_acc, outputs=(acc, bonus, None))

    def step(sel=None):
        for i in range(gamma):
            decode(i, sel)
        verify()
        accept()

    # eager reference step, then capture the step once in a HIP graph
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    ref = (out_dec.clone(), out_ver.clone(), acc.clone(), bonus.clone())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for r in range(3):                                            # every replay matches the eager step
        graph.replay()
        torch.cuda.synchronize()
        got = (out_dec, out_ver, acc, bonus)
        for a, b in zip(got, ref):
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.int16) if b.dtype == torch.bfloat16 else b), f"graph replay {r}"
        step()                                                    # eager work between replays
        torch.cuda.synchronize()
    planted = [x[3] for x in lg]
    assert acc.cpu().tolist() == planted, "accept lengths differ from the planted prefixes"

    log(f"timing {args.steps} graph replays after {args.warmup} warm-up")
    for _ in range(args.warmup):
        graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    us_step = wall * 1e6 / args.steps

    # spread: every replay between its own pair of events, outside the timed region above
    per = []
    for _ in range(max(args.steps, 100)):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        graph.replay()
        b.record()
        per.append((a, b))
    torch.cuda.synchronize()
    per = np.array([a.elapsed_time(b) * 1e3 for a, b in per])
    pct = {"p10": round(float(np.percentile(per, 10)), 2), "median": round(float(np.median(per)), 2),
           "p90": round(float(np.percentile(per, 90)), 2), "replays": int(per.size)}

    # the same step at the workload's other budget (its own selection and graph)
    graph2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph2):
        step((idx2, nsel2))
    for _ in range(args.warmup):
        graph2.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph2.replay()
    torch.cuda.synchronize()
    us_step2 = (time.perf_counter() - t0) * 1e6 / args.steps

    # per-kernel durations: one HIP graph of back-to-back launches per kernel, replayed after an
    # identical replay so the queue is busy when the start event is recorded; the events sit on
    # the stream the kernels run on
    log("timing kernels one by one")

    def graph_of(fn, n):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(n):
                fn()
        return g

    def time_graph(g, n, reps=5):
        vals = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            g.replay()
            a.record()
            g.replay()
            b.record()
            torch.cuda.synchronize()
            vals.append(a.elapsed_time(b) * 1e3 / n)
        return float(np.median(vals))

    n_dec = 10 * gamma
    kern_us = {
        "sparse_decode_attn": time_graph(graph_of(lambda: [decode(i) for i in range(gamma)], 10), n_dec),
        "verify_attn": time_graph(graph_of(verify, 10), 10),
        "accept_len": time_graph(graph_of(accept, 20), 20),
    }
    # cold: each launch right after a 512 MiB streaming read (more than the 256 MB MALL holds, as the
    # first draft of a step follows the verifier's 537 MB stream): time(graph of flush + op pairs) -
    # time(graph of flushes), per launch
    log("timing kernels cold (each after a 512 MiB read)")
    flush = cold_flush(torch, dev)
    n_cold = 10
    t_flush = time_graph(graph_of(flush, n_cold), n_cold)
    kern_us_cold = {}
    for name, fn in (("sparse_decode_attn", lambda: decode(0)), ("verify_attn", verify), ("accept_len", accept)):
        kern_us_cold[name] = time_graph(graph_of(lambda: (flush(), fn()), n_cold), n_cold) - t_flush
    del flush

    dec_b, ver_b, acc_b = algorithmic_bytes(S, Hq, Hkv, L, B, gamma, V)
    step_bytes = gamma * dec_b + ver_b + acc_b
    dec2_b = algorithmic_bytes(S, Hq, Hkv, L, B2, gamma, V)[0]
    step2_bytes = gamma * dec2_b + ver_b + acc_b
    kbytes = {"sparse_decode_attn": dec_b, "verify_attn": ver_b, "accept_len": acc_b}
    gbs = lambda n, us: round(kbytes[n] / (us * 1e-6) / 1e9, 1)
    frac = lambda n, us: round(kbytes[n] / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
    src_hash = hashlib.sha256(open(os.path.join(ROOT, "paper_2606_00144_amd", "csrc", "attn.hip"), "rb").read()).hexdigest()
    ver_gbs = ver_b / (kern_us["verify_attn"] * 1e-6) / 1e9
    roofline = {"bound": "hbm", "kernel": "verify_attn", "achieved": round(ver_gbs, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(ver_gbs / HBM_PEAK_GBS, 4), "traffic": traffic_from_profile(src_hash),
                "bytes_per_launch": ver_b, "avg_us": round(kern_us["verify_attn"], 2)}

    result = {
        "metric": METRIC, "value": round(us_step, 2), "unit": "us/step", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(us_step / 1e3, 5),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 K/V/Q with 0.5% planted heavy hitters; planted-argmax fp32 logits)",
        "config": {"workload": "16k-collapse-b8: 8 seqs x 16384 ctx, 32 q heads / 8 kv heads x 128, "
                               f"B={B}, gamma={gamma}, vocab {V}, separate drafter and verifier caches",
                   "num_seqs": S, "seq_len": L, "budget": B, "gamma": gamma, "vocab": V},
        "step_gbps": round(step_bytes / (us_step * 1e-6) / 1e9, 1),
        "step_bytes": step_bytes,
        "kernels_us": {n: round(v, 2) for n, v in kern_us.items()},
        "step_us_spread": pct,
        "kernels_gbps": {n: gbs(n, v) for n, v in kern_us.items()},
        "kernels_us_cold": {n: round(v, 2) for n, v in kern_us_cold.items()},
        "kernels_gbps_cold": {n: gbs(n, v) for n, v in kern_us_cold.items()},
        "targets_60pct_hbm": {n: {"frac_warm": frac(n, kern_us[n]), "frac_cold": frac(n, kern_us_cold[n]),
                                  "met_warm": frac(n, kern_us[n]) >= 0.6, "met_cold": frac(n, kern_us_cold[n]) >= 0.6}
                              for n in ("sparse_decode_attn", "verify_attn")},
        f"step_b{B2}": {"value": round(us_step2, 2), "unit": "us/step", "step_bytes": step2_bytes,
                        "step_gbps": round(step2_bytes / (us_step2 * 1e-6) / 1e9, 1)},
        "roofline": roofline,
        "cpu_baseline": None,
        # context only, not comparable: the paper's whole-model end-to-end speedups over AR decoding
        "paper_context": {"speedup_vs_ar_end_to_end": {"4K": 6.55, "8K": 4.46, "16K": 2.10},
                          "hardware": "one NVIDIA A100 80GB", "scope": "whole 7B verifier + 68M drafter, prefill included",
                          "source": "Sec. 4 main results"},
    }
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on the host (one step)")
        result["cpu_baseline"] = cpu_baseline(host, S, Hq, L, B, gamma)
    print(json.dumps(result), flush=True)


def cold_flush(torch, dev):
    """A launch that streams 512 MiB through the memory hierarchy and leaves little dirty data: one
    float of every 64-byte sector of a 512 MiB buffer copied to a 32 MiB one (an elementwise copy,
    graph-capturable).  More than the 256 MB MALL is read, so the next kernel finds none of its inputs
    there; a write flush instead would leave its dirty lines to be written back during that kernel."""
    src = torch.ones((128 << 20,), dtype=torch.float32, device=dev)
    dst = torch.empty((8 << 20,), dtype=torch.float32, device=dev)
    return lambda: dst.copy_(src[::16])


def _bf(torch, np, bits, dev):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)


def _time_calls(torch, fn, steps, warmup):
    """Mean µs per call over `steps` back-to-back eager calls (events on the calls' stream)."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e3 / steps


def _time_graph(torch, fn, steps, warmup, per_graph=1):
    """Mean µs per call of `fn`: `per_graph` calls captured once in a HIP graph, replayed back to back
    (launch latency of the small kernels is what a serving loop sees; no host work between replays).
    Several calls per graph keep the gap between graph replays out of a short kernel's time."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(per_graph):
            fn()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        graph.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e3 / (steps * per_graph)


def bench_select(args, bd, synth, torch, np, dev):
    """bd_select_kv on the 16K batch (8 x 16,384, W = 32, pool 7, B = --budget)."""
    cfg = synth.workload("16k-collapse-b8")
    S, Hq, Hkv, L, W, B = cfg.num_seqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.seq_len, cfg.window, args.budget
    log("generating inputs")
    qs, kS, _ = synth.kv_batch(cfg)
    k = _bf(torch, np, np.stack(kS), dev)
    q_win = _bf(torch, np, np.stack(qs)[:, -W:], dev)
    lens = torch.full((S,), L, dtype=torch.int32, device=dev)
    ws = bd.Workspace()
    steps = max(1, min(args.steps, 50))
    if args.chunk > 0:
        fn = lambda: bd.bd_select_kv_chunks(k, q_win, lens, B, chunk=args.chunk, workspace=ws)
    else:
        fn = lambda: bd.bd_select_kv(k, q_win, lens, B, workspace=ws)
    us = _time_calls(torch, fn, steps, min(args.warmup, 5))
    # the one-pass variant: the window rows' log-sum-exps given (the drafter's prefill attention produces
    # them), so only the second scoring pass reads K; formed here in fp32 outside the timed region
    G = Hq // Hkv
    lse = torch.empty((S, W, Hq), dtype=torch.float32, device=dev)
    pos = torch.arange(L, device=dev)
    for si in range(S):
        for g in range(Hkv):
            qf = q_win[si, :, g * G:(g + 1) * G].float().reshape(W * G, 128)          # rows (i, h)
            lg = (qf @ k[si, g].float().T) * (1.0 / 128 ** 0.5)
            rp = (L - W + torch.arange(W, device=dev)).repeat_interleave(G)
            lg = lg.masked_fill(pos[None, :] > rp[:, None], float("-inf"))
            lse[si, :, g * G:(g + 1) * G] = torch.logsumexp(lg, dim=1).reshape(W, G)
    if args.chunk > 0:
        fn1 = lambda: bd.bd_select_kv_chunks(k, q_win, lens, B, chunk=args.chunk, lse_win=lse, workspace=ws)
    else:
        fn1 = lambda: bd.bd_select_kv(k, q_win, lens, B, lse_win=lse, workspace=ws)
    us1 = _time_calls(torch, fn1, steps, min(args.warmup, 5))
    policy = f"TopKChunks s={args.chunk}" if args.chunk > 0 else "pool 7"
    alg = S * Hkv * L * 128 * 2 + S * W * Hq * 128 * 2 + S * Hkv * B * 4     # K once, window queries, idx
    gbs = alg / (us * 1e-6) / 1e9
    print(json.dumps({
        "metric": f"bd_select_kv µs/call and HBM GB/s at 16K ctx (8 seqs, W=32, {policy})", "value": round(us, 2),
        "unit": "us/call", "n_gpus": 1, "steps": steps, "warmup": min(args.warmup, 5),
        "ms_per_step": round(us / 1e3, 5), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded N(0,1) bf16 K/Q with 0.5% planted heavy hitters)",
        "config": {"workload": f"select-16k-b8: 8 seqs x {L} ctx, {Hq}/{Hkv} heads, W={W}, B={B}, {policy}",
                   "num_seqs": S, "seq_len": L, "budget": B},
        "roofline": {"bound": "hbm", "kernel": "bd_select_kv (two scoring passes + top-B)",
                     "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None, "bytes_per_call": alg},
        "one_pass_with_lse_win": {"value": round(us1, 2), "unit": "us/call",
                                  "gbps": round(alg / (us1 * 1e-6) / 1e9, 1)},
    }), flush=True)


def _multiview_inputs(bd, synth, torch, np, dev, name="multiview-train-b4-8k"):
    """The multi-view block and its views: the 4 x 8,192 block (C = 64, four sampled budgets, views from
    bd_select_kv), or the training shape (1 x 16,384, C = 256, the TopKChunks views of every training
    budget: top floor(B/8) prefix chunks with the block on top)."""
    cfg = synth.workload(name)
    S, Hq, Hkv, L, C = cfg.num_seqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.seq_len, cfg.block_len
    chunks = name == "train-c256-16k"
    budgets = list(cfg.budgets) if chunks else [int(b) for b in synth.view_budgets(cfg)]
    log("generating inputs")
    qs, ks, vs = synth.kv_batch(cfg)
    k, v = _bf(torch, np, np.stack(ks), dev), _bf(torch, np, np.stack(vs), dev)
    q_blk = _bf(torch, np, np.stack(qs)[:, -C:], dev)
    lens = torch.full((S,), L, dtype=torch.int32, device=dev)
    ld = max(budgets) + (C if chunks else 0)
    idx = torch.full((len(budgets), S, Hkv, ld), -1, dtype=torch.int32, device=dev)
    nsel = torch.empty((len(budgets), S), dtype=torch.int32, device=dev)
    for i, Bv in enumerate(budgets):                       # each view is the selection at its budget
        if chunks:
            vi, vn = bd.bd_select_kv_chunks(k, q_blk, lens, Bv, chunk=8)
        else:
            vi, vn = bd.bd_select_kv(k, q_blk, lens, Bv)
        idx[i, :, :, :vi.shape[2]] = vi
        nsel[i] = vn
    return cfg, budgets, k, v, q_blk, lens, idx, nsel


def _visible_pairs(np, idx_h, nsel_h, S, Hkv, G, L, C):
    """(query row, visible key) pairs over all branches, and those whose key is a block row."""
    pos = np.arange(L - C, L)
    full_pairs = S * Hkv * G * int((pos + 1).sum())
    blk_pairs = S * Hkv * G * (C * (C + 1) // 2)
    view_pairs = 0
    for i in range(idx_h.shape[0]):
        for s in range(S):
            for g in range(Hkv):
                t = idx_h[i, s, g, :nsel_h[i, s]]
                t = np.sort(t[(t >= 0) & (t < L)])
                view_pairs += G * int(np.searchsorted(t, pos, side="right").sum())
                tb = t[t >= L - C] - (L - C)                  # block keys listed in the view
                blk_pairs += G * int((C - tb).sum())
    return full_pairs + view_pairs, blk_pairs


def bench_multiview(args, bd, synth, torch, np, dev):
    """bd_multiview_attn on the multi-view block (4 x 8,192, C = 64, four budgets, views from bd_select_kv),
    or on the training shape (--mv-workload train-c256-16k)."""
    cfg, budgets, k, v, q_blk, lens, idx, nsel = _multiview_inputs(bd, synth, torch, np, dev, args.mv_workload)
    S, Hq, Hkv, L, C = cfg.num_seqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.seq_len, cfg.block_len
    ws = bd.Workspace()
    steps = max(1, min(args.steps, 50))
    fn = lambda: bd.bd_multiview_attn(k, v, q_blk, idx, nsel, lens, workspace=ws)
    us = _time_calls(torch, fn, steps, min(args.warmup, 5))
    # algorithmic flops: 4 * 128 per (query row, visible key), full branch and every view
    pairs, _ = _visible_pairs(np, idx.cpu().numpy(), nsel.cpu().numpy(), S, Hkv, Hq // Hkv, L, C)
    flops = 4 * 128 * pairs
    tflops = flops / (us * 1e-6) / 1e12
    print(json.dumps({
        "metric": f"bd_multiview_attn µs/call at {L // 1024}K ctx ({S} seqs, C={C}, {len(budgets)} views + full)",
        "value": round(us, 2),
        "unit": "us/call", "n_gpus": 1, "steps": steps, "warmup": min(args.warmup, 5),
        "ms_per_step": round(us / 1e3, 5), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded N(0,1) bf16 K/V/Q with 1% planted heavy hitters)",
        "config": {"workload": f"{cfg.name}: {S} seqs x {L} ctx, {Hq}/{Hkv} heads, C={C}, budgets {budgets}",
                   "num_seqs": S, "seq_len": L, "block_len": C, "budgets": budgets},
        "roofline": {"bound": "mfma", "kernel": "block_kernel (views + full branch)", "achieved": round(tflops, 1),
                     "peak": 2500.0, "unit": "TFLOP/s", "frac": round(tflops / 2500.0, 4), "traffic": None,
                     "flops_per_call": flops},
    }), flush=True)


def bench_multiview_bwd(args, bd, synth, torch, np, dev):
    """bd_multiview_attn_bwd on the multi-view block (or the training shape): dQ over every branch, dK/dV of
    the block rows."""
    cfg, budgets, k, v, q_blk, lens, idx, nsel = _multiview_inputs(bd, synth, torch, np, dev, args.mv_workload)
    S, Hq, Hkv, L, C = cfg.num_seqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.seq_len, cfg.block_len
    ov, of, o32v, lv, o32f, lf = bd.bd_multiview_attn(k, v, q_blk, idx, nsel, lens, train=True)
    g = torch.Generator(device=dev)
    g.manual_seed(3)
    dov = torch.randn(ov.shape, device=dev, generator=g).to(torch.bfloat16)
    dof = torch.randn(of.shape, device=dev, generator=g).to(torch.bfloat16)
    ws = bd.Workspace()
    steps = max(1, min(args.steps, 50))
    fn = lambda: bd.bd_multiview_attn_bwd(k, v, q_blk, idx, nsel, lens, o32v, lv, dov, o32f, lf, dof, workspace=ws)
    us = _time_calls(torch, fn, steps, min(args.warmup, 5))
    # algorithmic flops: per (query row, visible key) the score, dP and dQ products (6 * 128); per
    # (query row, visible block key) also the dK and dV products (4 * 128)
    pairs, blk = _visible_pairs(np, idx.cpu().numpy(), nsel.cpu().numpy(), S, Hkv, Hq // Hkv, L, C)
    flops = 6 * 128 * pairs + 4 * 128 * blk
    tflops = flops / (us * 1e-6) / 1e12
    print(json.dumps({
        "metric": f"bd_multiview_attn_bwd µs/call at {L // 1024}K ctx ({S} seqs, C={C}, {len(budgets)} views + full)",
        "value": round(us, 2),
        "unit": "us/call", "n_gpus": 1, "steps": steps, "warmup": min(args.warmup, 5),
        "ms_per_step": round(us / 1e3, 5), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded N(0,1) bf16 K/V/Q/dO with 1% planted heavy hitters)",
        "config": {"workload": f"{cfg.name}: {S} seqs x {L} ctx, {Hq}/{Hkv} heads, C={C}, budgets {budgets}",
                   "num_seqs": S, "seq_len": L, "block_len": C, "budgets": budgets},
        "roofline": {"bound": "mfma", "kernel": "dq_kernel + dkv_kernel", "achieved": round(tflops, 1),
                     "peak": 2500.0, "unit": "TFLOP/s", "frac": round(tflops / 2500.0, 4), "traffic": None,
                     "flops_per_call": flops},
    }), flush=True)


def bench_paged(args, bd, synth, torch, np, dev):
    """Verify and sparse decode on the ragged paged batch: 64 MHA sequences (32 heads) of 4K-16K tokens in
    16-token pages under a seeded page table, gamma = 5, B = 1024 (the selection over the pool runs once,
    untimed).  Each call warm (back-to-back) and cold (after a 512 MiB write)."""
    cfg = synth.workload("ragged-paged-b64-mha")
    S, Hq, Hkv, W, gamma, B, P = (cfg.num_seqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.window, cfg.gamma,
                                  cfg.budgets[0], cfg.page_size)
    lens_h = synth.seq_lens(cfg)
    log("generating inputs (64 sequences)")
    qs, ks, vs = synth.kv_batch(cfg, workers=16)
    table, npages = synth.page_table(cfg, lens_h)
    pool_k = np.zeros((npages, Hkv, P, 128), np.uint16)
    pool_v = np.zeros_like(pool_k)
    for s, L in enumerate(lens_h):
        for pi in range((int(L) + P - 1) // P):
            n = min(P, int(L) - pi * P)
            pool_k[table[s, pi], :, :n] = ks[s][:, pi * P:pi * P + n]
            pool_v[table[s, pi], :, :n] = vs[s][:, pi * P:pi * P + n]
    del ks, vs
    kd, vd = _bf(torch, np, pool_k, dev), _bf(torch, np, pool_v, dev)
    del pool_k, pool_v
    pt = torch.from_numpy(table).to(dev)
    lens = torch.from_numpy(lens_h.astype(np.int32)).to(dev)
    q_tail = _bf(torch, np, np.stack(qs), dev)
    q_win = q_tail[:, -W:].contiguous()
    q_dec = q_tail[:, -1].contiguous()
    q_ver = q_tail[:, -(gamma + 1):].contiguous()
    idx, nsel = bd.bd_select_kv(kd, q_win, lens, B, page_table=pt)
    out_d, out_v = torch.empty_like(q_dec), torch.empty_like(q_ver)
    ws_d, ws_v = bd.Workspace(), bd.Workspace()
    dec = lambda: bd.bd_sparse_decode_attn(kd, vd, q_dec, idx, nsel, lens, page_table=pt, out=out_d, workspace=ws_d)
    ver = lambda: bd.bd_verify_attn(kd, vd, q_ver, lens, page_table=pt, out=out_v, workspace=ws_v)
    torch.cuda.synchronize()
    steps, warm = max(1, min(args.steps, 50)), min(args.warmup, 5)
    us = {"verify_attn": _time_graph(torch, ver, steps, warm, 4), "sparse_decode_attn": _time_graph(torch, dec, steps, warm, 10)}
    flush = cold_flush(torch, dev)
    t_flush = _time_graph(torch, flush, steps, warm, 4)
    us_cold = {"verify_attn": _time_graph(torch, lambda: (flush(), ver()), steps, warm, 4) - t_flush,
               "sparse_decode_attn": _time_graph(torch, lambda: (flush(), dec()), steps, warm, 4) - t_flush}
    D = 128
    nb = {"verify_attn": int(lens_h.sum()) * Hkv * D * 2 * 2 + 2 * S * (gamma + 1) * Hq * D * 2,
          "sparse_decode_attn": S * Hkv * min(B, int(lens_h.min())) * (D * 2 * 2 + 4) + 2 * S * Hq * D * 2}
    g = lambda n, t: round(nb[n] / (t * 1e-6) / 1e9, 1)
    vb = g("verify_attn", us["verify_attn"])
    print(json.dumps({
        "metric": "ragged paged batch: verify and sparse decode µs/call and HBM GB/s (64 MHA seqs, 4K-16K ctx)",
        "value": round(us["verify_attn"], 2), "unit": "us/call (verify)", "n_gpus": 1, "steps": steps, "warmup": warm,
        "ms_per_step": round(us["verify_attn"] / 1e3, 5), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded N(0,1) bf16 K/V/Q with 1% planted heavy hitters)",
        "config": {"workload": f"ragged-paged-b64-mha: {S} seqs, ctx {int(lens_h.min())}-{int(lens_h.max())} "
                               f"(mean {float(lens_h.mean()):.0f}), {Hq}/{Hkv} heads, pages of {P}, B={B}, gamma={gamma}",
                   "num_seqs": S, "budget": B, "gamma": gamma, "page_size": P},
        "kernels_us": {n: round(t, 2) for n, t in us.items()},
        "kernels_gbps": {n: g(n, t) for n, t in us.items()},
        "kernels_us_cold": {n: round(t, 2) for n, t in us_cold.items()},
        "kernels_gbps_cold": {n: g(n, t) for n, t in us_cold.items()},
        "bytes_per_call": nb,
        "roofline": {"bound": "hbm", "kernel": "verify_attn (paged)", "achieved": vb, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(vb / HBM_PEAK_GBS, 4), "traffic": None,
                     "bytes_per_launch": nb["verify_attn"]},
    }), flush=True)


def bench_updates(args, bd, synth, torch, np, dev):
    """One round of Alg. 2's cache updates on the 16K batch: gamma single-row appends to the drafter
    cache and its sparse list, gamma+1 rows to the verifier cache, then both rollbacks (accept = 0,
    so every round leaves each cache one row longer)."""
    cfg = synth.workload("16k-collapse-b8")
    S, Hq, Hkv, L, gamma, B = cfg.num_seqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.seq_len, cfg.gamma, args.budget
    steps = max(1, min(args.steps, 50))
    warm = min(args.warmup, 5)
    cap = L + steps + warm + 4
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    kS = torch.randn((S, Hkv, cap, 128), device=dev, generator=g).to(torch.bfloat16)
    vS, kL, vL = torch.empty_like(kS), torch.empty_like(kS), torch.empty_like(kS)
    lensS = torch.full((S,), L - gamma - 1, dtype=torch.int32, device=dev)
    lensL = lensS.clone()
    idx = torch.zeros((S, Hkv, B + gamma * (steps + warm + 2)), dtype=torch.int32, device=dev)
    nsel = torch.full((S,), B, dtype=torch.int32, device=dev)
    rows1 = torch.randn((S, 1, Hkv, 128), device=dev, generator=g).to(torch.bfloat16)
    rowsV = torch.randn((S, gamma + 1, Hkv, 128), device=dev, generator=g).to(torch.bfloat16)
    acc = torch.zeros((S,), dtype=torch.int32, device=dev)

    def round_():
        for _ in range(gamma):
            bd.bd_cache_append(kS, vS, lensS, rows1, rows1, idx=idx, nsel=nsel)
        bd.bd_cache_append(kL, vL, lensL, rowsV, rowsV)
        bd.bd_cache_rollback(lensL, acc, gamma)
        bd.bd_cache_rollback(lensS, acc, gamma - 1, nsel=nsel)

    us = _time_graph(torch, round_, steps, warm)
    moved = 2 * (gamma + gamma + 1) * S * Hkv * 128 * 2 * 2        # rows read and written, K and V
    print(json.dumps({
        "metric": "Alg. 2 cache updates µs/round at 16K ctx (8 seqs: 5 drafter appends, 1 verifier append, 2 rollbacks)",
        "value": round(us, 2), "unit": "us/round", "n_gpus": 1, "steps": steps, "warmup": warm,
        "ms_per_step": round(us / 1e3, 5), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (random rows)",
        "config": {"workload": f"updates-16k-b8: 8 seqs, {Hkv} kv heads, gamma={gamma}, B={B}", "num_seqs": S,
                   "seq_len": L, "gamma": gamma},
        "roofline": {"bound": "latency", "kernel": "append_rows/append_advance/rollback (9 launches per round)",
                     "achieved": round(moved / (us * 1e-6) / 1e9, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(moved / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 6), "traffic": None,
                     "bytes_per_round": moved},
    }), flush=True)


def bench_ce(args, bd, synth, torch, np, dev):
    """Top-1 CE with the targets' scan fused (Eqs. 5-7) on the multi-view training shape: the 4 x 64
    continuation rows, vocabulary 32,000; student and teacher logits fp32."""
    cfg = synth.workload("multiview-train-b4-8k")
    R, V = cfg.num_seqs * cfg.block_len, 32000
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    student = torch.randn((R, V), device=dev, generator=g) * 2
    teacher = torch.randn((R, V), device=dev, generator=g) * 2
    ws = bd.Workspace()
    steps, warm = max(1, min(args.steps, 100)), min(args.warmup, 10)
    per_graph = 10
    us = _time_graph(torch, lambda: bd.bd_top1_ce(student, teacher=teacher, workspace=ws), steps, warm, per_graph)
    alg = 2 * R * V * 4 + R * 4
    gbs = alg / (us * 1e-6) / 1e9
    print(json.dumps({
        "metric": "top-1 CE (fused teacher argmax) µs/call and HBM GB/s, 256 rows x 32,000 vocab",
        "value": round(us, 2), "unit": "us/call", "n_gpus": 1, "steps": steps, "warmup": warm,
        "ms_per_step": round(us / 1e3, 5), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "fp32", "data": "synthetic (N(0, 4) logits)", "calls_per_graph": per_graph,
        "config": {"workload": f"ce-train-b4: {R} rows (4 seqs x C={cfg.block_len}), vocab {V}", "rows": R, "vocab": V},
        "roofline": {"bound": "hbm", "kernel": "ce_kernel", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None, "bytes_per_call": alg},
    }), flush=True)


if __name__ == "__main__":
    main()
