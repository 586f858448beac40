#!/usr/bin/env python3
"""Benchmark of exact top-k context-sparse decode attention on one MI355X.

One step = one fused sparse_decode_attention call over a whole decode batch:
score every cached key, keep the exact top-k per query head, gather and
attend.  Default workload: batch 16, 64 query / 8 KV heads, d = 128,
N = 131072 (128K) cached positions per sequence, bfloat16, 100x sparsity
(k = 1311), a 64-token high-norm prefix and 1% planted high-similarity keys;
synthetic, seeded.  Inputs are resident in HBM before timing starts.

Prints one JSON line: queries/s (decode queries per second) as the value,
the achieved HBM bandwidth of the whole path and of its dominant kernel (the
scoring stream) against the 8 TB/s peak, and the CPU oracle timed on a
bounded sample of the same workload on this host.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "sparse decode attention: queries/sec + achieved HBM GB/s vs peak at N=128K"
COUNTERS_FILE = os.path.join(ROOT, "profiles", "score_stream_w3_counters.json")
KERNEL_SRC = [os.path.join(ROOT, "paper_2605_24168_amd", "csrc", f)
              for f in ("sd_kernels.hip", "sd_internal.hpp")]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_hash() -> str:
    """Hash of the kernel sources (counters taken on other sources are stale)."""
    h = hashlib.sha256()
    for path in KERNEL_SRC:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def path_bytes(inp, ks, labels=False, samples=0):
    """Algorithmic HBM bytes of one step: every key (or, with the label
    indexer, every 16-byte label row) once, the kept value rows, q, out and
    idx.  (Per-head mode gathers one value row per query head and kept
    position, plus its key row when the attention recomputes its logits:
    forced positions or label selection; group-shared mode one key and one
    value row per KV head.)"""
    e = 2 if inp.dtype == "bf16" else 4
    row = inp.d * e
    key_stream = sum(int(L) for L in inp.seq_lens) * inp.Hkv * (16 if labels else row)
    if inp.group_shared:
        gather = sum(int(k) for k in ks) * inp.Hkv * 2 * row
    else:
        recompute = labels or inp.n_sink + inp.n_local > 0 or samples > 0
        per_entry = 2 * row if recompute else row
        gather = sum(int(k) + samples for k in ks) * inp.Hq * per_entry
    k_max = max(int(k) for k in ks) + samples
    small = 2 * inp.B * inp.Hq * row + inp.B * inp.rows * k_max * 4
    return key_stream, gather, small


def union_gather_rows(torch, idx, inp):
    """Distinct (KV head, position) pairs of a step's index lists: the value
    rows a group-deduplicated gather would read (per-head mode lists the
    same position once per query head that keeps it)."""
    if inp.group_shared or inp.G == 1:
        return int((idx >= 0).sum().item())
    s = idx.view(inp.B, inp.Hkv, -1).sort(dim=-1).values
    first = torch.ones_like(s, dtype=torch.bool)
    first[..., 1:] = s[..., 1:] != s[..., :-1]
    return int(((s >= 0) & first).sum().item())


def read_peak(torch, sd, gib=4, reps=10):
    """Median rate of a plain streaming read of a gib-GiB device buffer
    (the library's read probe), GB/s."""
    buf = torch.zeros(gib << 30, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    for _ in range(2):
        sd.read_probe(buf, sink)
    ms = []
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        sd.read_probe(buf, sink)
        e1.record()
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1))
    del buf
    ms.sort()
    return (gib << 30) / (ms[len(ms) // 2] * 1e-3) / 1e9


def flushed_calls(torch, fn, n, flush_gib=1):
    """n calls, each timed alone by events around it, with a flush_gib-GiB
    buffer written before each (outside the events) so that no cache holds
    the previous call's data.  Returns (median, p10, p90) in ms."""
    flush = torch.empty(flush_gib << 30, dtype=torch.uint8, device="cuda")
    ms = []
    for _ in range(n):
        flush.zero_()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1))
    del flush
    ms.sort()
    pick = lambda f: ms[min(len(ms) - 1, int(round(f * (len(ms) - 1))))]
    return pick(0.5), pick(0.1), pick(0.9)


def flushed_loop(torch, fn, n, flush_gib=1, reps=3):
    """Per-call time after a cache flush without per-call events: (flush,
    call) n times between two events, minus n flushes alone; the best of
    reps.  Returns ms per call."""
    flush = torch.empty(flush_gib << 30, dtype=torch.uint8, device="cuda")

    def loop(with_call):
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            flush.zero_()
            if with_call:
                fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    both = min(loop(True) for _ in range(reps))
    alone = min(loop(False) for _ in range(reps))
    del flush
    return both - alone


def extra_workload(args, cfg):
    """Another workload measured the same way as the default line's (back to
    back steps, the scoring kernel's launches, per-call times after a cache
    flush), without the CPU oracle leg.  Returns a dict for the JSON line."""
    import torch
    from paper_2605_24168_amd import sparse_decode as sd
    from paper_2605_24168_amd import synth

    log(f"generating workload {cfg} ({synth.NAMES[cfg]})")
    inp = synth.make_inputs(cfg, seed=args.seed)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    ks = [sd.budget(int(L), sp) for L in inp.seq_lens]
    k_max = sd.k_max_of(cache, sp)
    out = torch.empty_like(q)
    idx = torch.empty((inp.B, inp.rows, k_max), dtype=torch.int32, device="cuda")
    ws = torch.empty(sd.workspace_size(q, cache, sp, idx), dtype=torch.uint8, device="cuda")
    sd.set_workspace(ws)
    fn = lambda: sd.sparse_decode_attention(q, cache, lens, sp, out=out, idx=idx)
    log(f"workload {cfg}: warmup {args.warmup}, timing {args.steps} steps")
    for _ in range(args.warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        fn()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / args.steps * 1e3
    sd.set_profiling(2)
    for _ in range(args.steps):
        fn()
    torch.cuda.synchronize()
    sd.set_profiling(False)
    score_ms = sd.profile_mean()["score_ms"]
    sd.set_profiling(True)
    for _ in range(args.steps):
        fn()
    torch.cuda.synchronize()
    sd.set_profiling(False)
    prof = sd.profile_mean()
    med = p10 = p90 = loop_ms = None
    if args.calls > 0:
        log(f"workload {cfg}: {args.calls} calls one by one after a cache flush")
        med, p10, p90 = flushed_calls(torch, fn, args.calls)
        loop_ms = flushed_loop(torch, fn, args.calls)
    key_b, gather_b, small_b = path_bytes(inp, ks)
    total_b = key_b + gather_b + small_b
    rec = {
        "workload": synth.NAMES[cfg],
        "ms_per_step": ms,
        "queries_per_s": inp.B / (ms * 1e-3),
        "path": {"algorithmic_bytes": total_b, "key_stream_bytes": key_b,
                 "value_gather_bytes": gather_b,
                 "achieved_GBps": total_b / (ms * 1e-3) / 1e9,
                 "frac_of_peak": total_b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                 "stage_ms": {k_: round(prof[k_], 4) for k_ in
                              ("pilot_ms", "score_ms", "select_ms", "repair_ms", "attend_ms",
                               "total_ms")},
                 "repaired_rows_last_step": prof["repaired_rows"]},
        "score_stream": {"avg_launch_ms": score_ms,
                         "achieved_GBps": (key_b + q.numel() * q.element_size())
                         / (score_ms * 1e-3) / 1e9 if score_ms > 0 else None},
        "calls_after_flush": None if med is None else {
            "n": args.calls, "median_ms": med, "p10_ms": p10, "p90_ms": p90,
            "path_frac_of_peak_at_median": total_b / (med * 1e-3) / 1e9 / HBM_PEAK_GBPS,
            "loop_ms_per_call": loop_ms},
    }
    sd.set_workspace(None)
    del q, cache, lens, out, idx, ws
    torch.cuda.empty_cache()
    return rec


def counters_traffic():
    """HBM bytes per launch of the scoring kernel from committed rocprofv3
    counters, if they were taken on the current kernel source."""
    try:
        with open(COUNTERS_FILE) as f:
            c = json.load(f)
    except (OSError, ValueError):
        return None
    if c.get("kernel_source_sha256_16") != kernel_hash():
        return None
    return c.get("hbm_bytes_per_launch")


def cpu_baseline(inp, n_seq, k_max, fixed_k=None, labels=None, min_s=10.0, draws=None,
                 threads=None):
    import dataclasses
    from oracle import oracle as O
    bs = list(range(min(n_seq, inp.B)))
    if inp.layout == "paged":
        sub = dataclasses.replace(inp, B=len(bs), q=inp.q[bs], seq_lens=inp.seq_lens[bs],
                                  block_table=inp.block_table[bs])
    else:
        sub = dataclasses.replace(inp, B=len(bs), q=inp.q[bs], k=inp.k[bs], v=inp.v[bs],
                                  seq_lens=inp.seq_lens[bs])
    if threads is None:
        try:
            threads = len(os.sched_getaffinity(0))
        except AttributeError:
            threads = os.cpu_count() or 1
        threads = max(1, min(threads, 16))
    used = O.max_threads(threads)
    import numpy as np
    ko = None if fixed_k is None else np.full(len(bs), fixed_k, np.int32)

    def once():
        if draws is not None:
            O.sampled_attention(sub, draws[bs], k_max=k_max, k_override=ko, nthreads=threads)
        elif labels is None:
            O.sparse_attention(sub, k_max=k_max, k_override=ko, nthreads=threads)
        else:  # (label cache in the key cache's layout, channels)
            lab, ch = labels
            sub_lab = lab if inp.layout == "paged" else lab[bs]
            O.label_attention(sub, sub_lab, ch, k_max=k_max, k_override=ko, nthreads=threads)

    # The sample again and again until at least min_s of wall time: a
    # bounded, repeatable amount of CPU work whatever the sample size.
    reps, t0 = 0, time.perf_counter()
    while True:
        once()
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_s:
            break
    return {"value": reps * len(bs) / dt, "unit": "queries/s", "cores": used, "kind": "oracle",
            "sample": f"{len(bs)} of {inp.B} sequences ({len(bs) * inp.rows} rows), "
                      f"score+select+attend in float64, {reps} passes in {dt:.2f} s wall"}


# Table 1 of the paper (H100 80GB HBM3, FP16, GQA 32/8, d 128, page 16, NHD,
# 128K context): FlashInfer dense decode ms per batch size and the sparse
# backend's speedup over it per sparsity.  Context for the MI355X sweep, not
# a target of the same hardware.
TABLE1_RATIOS = [2, 4, 10, 20, 50, 100, 200, 500]
TABLE1_H100 = {
    1: (0.19, [0.32, 0.63, 1.45, 2.58, 5.57, 10.25, 11.05, 11.14]),
    4: (0.72, [0.33, 0.66, 1.64, 3.18, 7.45, 13.36, 24.25, 42.04]),
    8: (1.50, [0.38, 0.77, 1.90, 3.75, 8.88, 16.82, 29.64, 76.14]),
    16: (3.08, [0.45, 0.89, 2.21, 4.35, 10.54, 20.09, 37.32, 76.77]),
}


# Table 2 of the paper (H100, FP16, 128K, page 16): FlashInfer dense ms and
# the speedup of the sparse backend with an 8-channel 16-bit Double Sparsity
# indexer choosing the positions, GQA 32/8 and MHA 32/32.  Context only.
TABLE2_RATIOS = [2, 5, 10, 20, 50, 100]
TABLE2_H100 = {
    "gqa": {1: (0.19, [0.28, 0.56, 0.83, 1.12, 1.46, 1.65]),
            4: (0.72, [0.32, 0.67, 1.06, 1.52, 2.11, 2.45]),
            8: (1.50, [0.36, 0.75, 1.18, 1.68, 2.30, 2.66]),
            16: (3.08, [0.41, 0.85, 1.31, 1.82, 2.46, 2.81])},
    "mha": {1: (0.70, [0.91, 1.62, 2.18, 2.68, 3.14, 3.37]),
            4: (2.79, [1.02, 1.86, 2.56, 3.17, 3.74, 4.00]),
            8: (5.61, [1.12, 2.00, 2.71, 3.32, 3.86, 4.11]),
            16: (11.18, [1.22, 2.13, 2.84, 3.43, 3.94, 4.17])},
}


def time_calls(torch, fn, steps, warmup):
    """Mean ms per call over `steps` calls after `warmup`, by events on the
    current stream around the whole run (no event between calls)."""
    for _ in range(warmup):
        fn()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def time_graph(torch, fn, steps, warmup, replays=5):
    """Mean ms per call with `steps` calls captured in one HIP graph, replayed
    `replays` times back to back (kernel time without the host's per-call
    work; the replays overlap each graph's launch with the previous one's
    kernels); also returns whether the replay left the same output as the
    eager calls.  fn() returns its output tensor."""
    for _ in range(warmup):  # eager: also sizes the library workspace before capture
        ref = fn()
    torch.cuda.synchronize()
    ref = ref.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(steps):
            out = fn()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(replays):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    same = bool(torch.equal(out, ref))
    del g
    return e0.elapsed_time(e1) / (steps * replays), same


def backend_table(args):
    """Table 1's shape on one MI355X: dense decode attention against the
    weighted sparse backend on irregular index lists, batch 1/4/8/16, 128K
    context, GQA 32/8, paged NHD (page 16), bfloat16.  Prints one JSON line."""
    import torch
    from paper_2605_24168_amd import sparse_decode as sd
    from paper_2605_24168_amd import synth

    torch.cuda.set_device(0)
    N, Hq, Hkv, d = 131072, 32, 8, 128
    batches = [1, 4, 8, 16]
    log("drawing the 16 x 128K paged cache on the GPU")
    t = synth.backend_sweep_inputs(B=max(batches), N=N, Hq=Hq, Hkv=Hkv, seed=args.seed)
    torch.cuda.synchronize()
    rows = []
    for B in batches:
        q = t["q"][:B].contiguous()
        cache = sd.KVCache(k=t["k"], v=t["v"], layout="paged",
                           block_table=t["block_table"][:B].contiguous())
        lens = t["seq_lens"][:B].contiguous()
        out = torch.empty_like(q)
        dense_fn = lambda: sd.sparse_decode_dense_attention(q, cache, lens, out=out)
        dense_eager = time_calls(torch, dense_fn, args.steps, args.warmup)
        dense_ms, same = time_graph(torch, dense_fn, args.steps, args.warmup)
        dense_bytes = B * Hkv * N * d * 2 * 2 + 2 * B * Hq * d * 2
        entry = {"batch": B, "dense_ms": round(dense_ms, 4), "dense_eager_ms": round(dense_eager, 4),
                 "dense_GBps": round(dense_bytes / (dense_ms * 1e-3) / 1e9, 1),
                 "dense_frac_of_peak": round(dense_bytes / (dense_ms * 1e-3) / 1e9
                                             / HBM_PEAK_GBPS, 4),
                 "graph_replay_matches_eager": same,
                 "h100_flashinfer_ms": TABLE1_H100[B][0], "sparse": {}}
        log(f"B={B}: dense {dense_ms:.4f} ms ({entry['dense_GBps']} GB/s), "
            f"eager {dense_eager:.4f} ms")
        for i, S in enumerate(TABLE1_RATIOS):
            k = int(round(N / S))
            idx, w = synth.backend_sweep_sets(B * Hq, N, k, seed=args.seed)
            idx, w = idx.view(B, Hq, k), w.view(B, Hq, k)
            sp = sd.Sparsity(ratio=float(S))
            fn = lambda: sd.sparse_decode_attend_weighted(q, cache, lens, idx, w, sp, out=out)
            eager = time_calls(torch, fn, args.steps, args.warmup)
            ms, same = time_graph(torch, fn, args.steps, args.warmup)
            sparse_bytes = B * Hq * k * (2 * d * 2 + 8) + 2 * B * Hq * d * 2
            entry["graph_replay_matches_eager"] &= same
            entry["sparse"][f"{S}x"] = {
                "k": k, "ms": round(ms, 4), "eager_ms": round(eager, 4),
                "speedup": round(dense_ms / ms, 3),
                "eager_speedup": round(dense_eager / eager, 3),
                "GBps": round(sparse_bytes / (ms * 1e-3) / 1e9, 1),
                "h100_speedup": TABLE1_H100[B][1][i]}
            log(f"  {S}x (k={k}): {ms:.4f} ms (eager {eager:.4f}), speedup {dense_ms / ms:.2f}x "
                f"(H100: {TABLE1_H100[B][1][i]}x)")
            del idx, w
        rows.append(entry)
    rec = {
        "table": "sparse backend vs dense decode (Table 1 shape)",
        "steps": args.steps, "warmup": args.warmup,
        "config": {"q_heads": Hq, "kv_heads": Hkv, "head_dim": d, "context": N,
                   "layout": "paged NHD, page 16, random page order", "dtype": "bf16",
                   "index_lists": "uniform random distinct positions per query head, "
                                  "weights U[0.05, 3)"},
        "timing": "ms: K calls captured in one HIP graph, replayed 5 times back to back "
                  "between events (kernel time, as a kernel benchmark measures it); eager_ms: "
                  "K calls back to back through the Python binding (adds its per-call host "
                  "work)",
        "dense_bytes": "all K and V rows of the batch",
        "sparse_bytes": "per query head and kept position one K and one V row (256 B each), "
                        "its index and weight",
        "rows": rows,
    }
    print(json.dumps(rec), flush=True)


def indexer_table(args):
    """Table 2's shape on one MI355X: dense decode attention against the
    method with the 8-channel label indexer choosing the positions (label
    stream, exact top-k on label scores, attention on full keys and
    values), batch 1/4/8/16, 128K context, GQA 32/8 and MHA 32/32, paged NHD,
    bfloat16.  Prints one JSON line."""
    import torch
    from paper_2605_24168_amd import sparse_decode as sd
    from paper_2605_24168_amd import synth

    torch.cuda.set_device(0)
    N, Hq, d = 131072, 32, 128
    batches = [1, 4, 8, 16]
    modes = []
    for mode, Hkv in (("gqa", 8), ("mha", 32)):
        log(f"drawing the 16 x 128K paged cache ({mode}, {Hq}q/{Hkv}kv) on the GPU")
        t = synth.backend_sweep_inputs(B=max(batches), N=N, Hq=Hq, Hkv=Hkv, seed=args.seed)
        ch_np = synth.label_channels(Hkv, seed=args.seed)
        ch = torch.from_numpy(ch_np).cuda()
        # label cache: each KV head's label channels of every key (bf16 copies)
        # label cache [pages, Hkv, 16, 8]: each KV head's label channels of
        # every key (bf16 copies), head-major inside a page
        lab = torch.stack([t["k"][:, :, g, :].index_select(2, ch[g].long())
                           for g in range(Hkv)], dim=1).contiguous()
        labels = sd.Labels(t=lab, channels=ch)
        torch.cuda.synchronize()
        rows = []
        for B in batches:
            q = t["q"][:B].contiguous()
            cache = sd.KVCache(k=t["k"], v=t["v"], layout="paged",
                               block_table=t["block_table"][:B].contiguous())
            lens = t["seq_lens"][:B].contiguous()
            out = torch.empty_like(q)
            dense_fn = lambda: sd.sparse_decode_dense_attention(q, cache, lens, out=out)
            dense_ms, _ = time_graph(torch, dense_fn, args.steps, args.warmup)
            kv_bytes = B * Hkv * N * d * 2 * 2
            entry = {"batch": B, "dense_ms": round(dense_ms, 4),
                     "dense_GBps": round(kv_bytes / (dense_ms * 1e-3) / 1e9, 1),
                     "h100_flashinfer_ms": TABLE2_H100[mode][B][0], "indexed": {}}
            log(f"{mode} B={B}: dense {dense_ms:.4f} ms ({entry['dense_GBps']} GB/s)")
            for i, S in enumerate(TABLE2_RATIOS):
                sp = sd.Sparsity(ratio=float(S))
                k_max = sd.k_max_of(cache, sp)
                idx = torch.empty((B, Hq, k_max), dtype=torch.int32, device="cuda")
                ws = torch.empty(sd.workspace_size(q, cache, sp, idx), dtype=torch.uint8,
                                 device="cuda")
                sd.set_workspace(ws)
                fn = lambda: sd.sparse_decode_label_attention(q, cache, labels, lens, sp, out=out,
                                                              idx=idx)[0]
                eager = time_calls(torch, fn, args.steps, args.warmup)
                ms, same = time_graph(torch, fn, args.steps, args.warmup)
                sd.set_profiling(True)
                for _ in range(args.steps):
                    fn()
                torch.cuda.synchronize()
                sd.set_profiling(False)
                prof = sd.profile_mean()
                sd.set_workspace(None)
                del ws, idx
                entry["indexed"][f"{S}x"] = {
                    "k": int(round(N / S)), "ms": round(ms, 4), "eager_ms": round(eager, 4),
                    "speedup": round(dense_ms / ms, 3),
                    "h100_speedup": TABLE2_H100[mode][B][1][i],
                    "graph_replay_matches_eager": same,
                    "stage_ms": {k_: round(prof[k_], 4) for k_ in
                                 ("pilot_ms", "score_ms", "select_ms", "repair_ms",
                                  "attend_ms")},
                    "fallback_rows": prof["repaired_rows"]}
                log(f"  {S}x: {ms:.4f} ms, speedup {dense_ms / ms:.2f}x "
                    f"(H100: {TABLE2_H100[mode][B][1][i]}x), stages {entry['indexed'][f'{S}x']['stage_ms']}")
            rows.append(entry)
        modes.append({"mode": mode, "q_heads": Hq, "kv_heads": Hkv, "rows": rows})
        del t, lab, labels
        torch.cuda.empty_cache()
    rec = {
        "table": "label indexer + sparse attention vs dense decode (Table 2 shape)",
        "steps": args.steps, "warmup": args.warmup,
        "config": {"head_dim": d, "context": N, "layout": "paged NHD, page 16, random page order",
                   "dtype": "bf16", "labels": "8 bf16 channels per key, uniform random channels "
                                              "per KV head (uncalibrated)"},
        "timing": "ms: K calls captured in one HIP graph, replayed 5 times (kernel time); "
                  "stage_ms: events between the stages (profiling on)",
        "modes": modes,
    }
    print(json.dumps(rec), flush=True)


def oracle_table(args):
    """The CPU oracle alone on workloads 1 and 2 (whole batches), on one core
    and on every core it may use: one JSON line.  No GPU is touched."""
    from oracle import oracle as O
    from paper_2605_24168_amd import synth
    rows = []
    for cfg in (1, 2):
        inp = synth.make_inputs(cfg, seed=args.seed)
        for threads in (1, None):
            r = cpu_baseline(inp, inp.B, O.k_max_for(inp), min_s=3.0, threads=threads)
            r.update(workload=cfg, name=synth.NAMES[cfg],
                     ms_per_call=1e3 * inp.B / r["value"])
            log(f"oracle workload {cfg}, {r['cores']} core(s): {r['ms_per_call']:.1f} ms/call")
            rows.append(r)
    print(json.dumps({"table": "CPU oracle (score + select + attend, float64) per call",
                      "rows": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-sample", type=int, default=8,
                    help="sequences of the workload the CPU oracle is timed on (0: skip)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, copy this many MiB device to device once (a plain "
                         "copy of known size that scales hardware traffic counters)")
    ap.add_argument("--extra-workloads", default="4,5,2,1",
                    help="comma-separated workloads measured after the default line's, without "
                         "the CPU oracle leg, and reported under extra_workloads ('' to skip)")
    ap.add_argument("--calls", type=int, default=30,
                    help="calls timed one by one after a cache flush (median/p10/p90; 0: skip)")
    ap.add_argument("--sink", type=int, default=0,
                    help="forced first positions of every sequence (sink window)")
    ap.add_argument("--local", type=int, default=0,
                    help="forced last positions of every sequence (local window)")
    ap.add_argument("--ratio", type=float, default=None,
                    help="sparsity S (top-k budget round(L/S)) instead of the workload's")
    ap.add_argument("--fixed-k", type=int, default=None,
                    help="top-k budget K for every sequence instead of the ratio rule")
    ap.add_argument("--samples", type=int, default=0,
                    help="stochastic index selection: this many importance-weighted uniform "
                         "draws of the rest of each row beside its exact top-k")
    ap.add_argument("--labels", action="store_true",
                    help="select with the 8-channel label indexer (bf16 workloads) instead of "
                         "exact scores")
    ap.add_argument("--table2", action="store_true",
                    help="instead of the default line, sweep dense decode against the method "
                         "with the 8-channel label indexer in Table 2's shape (batch 1/4/8/16, "
                         "2x-100x, 128K, GQA 32/8 and MHA 32/32, paged)")
    ap.add_argument("--table1", action="store_true",
                    help="instead of the default line, sweep dense decode against the "
                         "weighted sparse backend in Table 1's shape (batch 1/4/8/16, "
                         "2x-500x, 128K, GQA 32/8, paged)")
    ap.add_argument("--oracle-cores", action="store_true",
                    help="instead of the default line, time the CPU oracle on workloads 1 and "
                         "2 on one core and on all cores (no GPU)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the method's data-parallel shards (sequences or KV "
              "heads) need no exchange, so only --gpus 1 is supported", file=sys.stderr)
        sys.exit(2)
    if args.oracle_cores:
        oracle_table(args)
        return
    if args.table1:
        backend_table(args)
        return
    if args.table2:
        indexer_table(args)
        return

    import numpy as np
    import torch
    from paper_2605_24168_amd import sparse_decode as sd
    from paper_2605_24168_amd import synth

    torch.cuda.set_device(0)
    log(f"generating workload {args.workload} ({synth.NAMES[args.workload]})")
    t0 = time.perf_counter()
    extra = {} if args.ratio is None else {"ratio": args.ratio}
    inp = synth.make_inputs(args.workload, seed=args.seed, n_sink=args.sink, n_local=args.local,
                            **extra)
    log(f"  generated in {time.perf_counter() - t0:.1f} s; copying to the GPU")
    q, cache, lens = sd.cache_from_inputs(inp)
    k_override = None
    if args.fixed_k is not None:
        k_override = torch.full((inp.B,), args.fixed_k, dtype=torch.int32, device="cuda")
    sp = sd.sparsity_from_inputs(inp, k_override=k_override)
    ks = []
    for L in inp.seq_lens:  # list entries per sequence: forced positions + top-k
        L = int(L)
        if args.fixed_k is None:
            ks.append(sd.budget(L, sp))  # the library's rule
        else:
            ns = min(inp.n_sink, L)
            nl = min(inp.n_local, L - ns)
            ks.append(ns + nl + min(args.fixed_k, L - ns - nl))
    k_max = sd.k_max_of(cache, sp) if args.fixed_k is None else max(ks)
    out = torch.empty_like(q)
    idx = torch.empty((inp.B, inp.rows, k_max + args.samples), dtype=torch.int32, device="cuda")
    draws = wts = None
    if args.samples > 0:
        if args.labels:
            raise SystemExit("--samples and --labels do not combine")
        g = torch.Generator(device="cuda").manual_seed(args.seed)
        draws = torch.randint(-2**31, 2**31 - 1, (inp.B, inp.rows, args.samples),
                              dtype=torch.int32, device="cuda", generator=g)
        wts = torch.empty(idx.shape, dtype=torch.float32, device="cuda")
    ws = torch.empty(sd.workspace_size(q, cache, sp, idx), dtype=torch.uint8, device="cuda")
    sd.set_workspace(ws)
    labels = host_labels = None
    if args.labels:
        ch = synth.label_channels(inp.Hkv, seed=args.seed)
        host_labels = (synth.label_cache(inp, ch), ch)
        lab = synth.label_cache_device_layout(inp, host_labels[0])
        labels = sd.Labels(t=torch.from_numpy(lab).view(torch.bfloat16).cuda(),
                           channels=torch.from_numpy(ch).cuda())
    torch.cuda.synchronize()

    def one_step():
        if draws is not None:
            sd.sparse_decode_sampled_attention(q, cache, lens, sp, draws, out=out, idx=idx,
                                               weights=wts)
        elif labels is None:
            sd.sparse_decode_attention(q, cache, lens, sp, out=out, idx=idx)
        else:
            sd.sparse_decode_label_attention(q, cache, labels, lens, sp, out=out, idx=idx)

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()

    def run_steps(n):
        for _ in range(n):
            one_step()

    # Timed region: K steps, uninstrumented (any HIP timing event adds about
    # 20 us per step to the path on this GPU, so none is recorded here).
    log(f"timing {args.steps} steps")
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    run_steps(args.steps)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall / args.steps * 1e3
    ms_events = ev0.elapsed_time(ev1) / args.steps

    # The same K steps again with the scoring kernel timed by HIP events
    # attached to each of its dispatches on the call's stream (the roofline's
    # kernel time), then with events between every stage (stage breakdown).
    log(f"timing the scoring kernel over {args.steps} more steps")
    sd.set_profiling(2)
    torch.cuda.synchronize()
    u0 = time.perf_counter()
    run_steps(args.steps)
    torch.cuda.synchronize()
    ms_timed_kernel = (time.perf_counter() - u0) / args.steps * 1e3
    sd.set_profiling(False)
    score_prof = sd.profile_mean()
    sd.set_profiling(True)
    run_steps(args.steps)
    torch.cuda.synchronize()
    sd.set_profiling(False)
    prof = sd.profile_mean()

    # Calls one by one, each after a cache flush (events around each call).
    calls = None
    if args.calls > 0:
        log(f"timing {args.calls} calls one by one after a cache flush")
        med, p10, p90 = flushed_calls(torch, one_step, args.calls)
        loop_ms = flushed_loop(torch, one_step, args.calls)
        calls = {"n": args.calls, "median_ms": med, "p10_ms": p10, "p90_ms": p90,
                 "queries_per_s_at_median": inp.B / (med * 1e-3),
                 "loop_ms_per_call": loop_ms,
                 "timing": "HIP events around each call on its stream; a 1 GiB device buffer "
                           "written before each call, outside the events.  loop_ms_per_call: "
                           "(flush, call) repeated between two events, minus the flushes "
                           "alone (no per-call events)"}
    union_rows = union_gather_rows(torch, idx, inp)

    # Dense decode attention over the same cache: the full-attention baseline.
    dense = None
    if inp.dtype == "bf16" and inp.G <= 8:
        log(f"timing dense decode attention over {args.steps} steps")
        dense_ms = time_calls(torch, lambda: sd.sparse_decode_dense_attention(q, cache, lens,
                                                                              out=out),
                              args.steps, args.warmup)
        dense_b = sum(int(L) for L in inp.seq_lens) * inp.Hkv * inp.d * 2 * 2
        dense = {"ms_per_step": dense_ms,
                 "GBps": dense_b / (dense_ms * 1e-3) / 1e9,
                 "frac_of_peak": dense_b / (dense_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                 "sparse_speedup": dense_ms / ms_step}

    key_b, gather_b, small_b = path_bytes(inp, ks, labels=args.labels, samples=args.samples)
    total_b = key_b + gather_b + small_b
    path_gbps = total_b / (ms_step * 1e-3) / 1e9
    q_bytes = inp.B * inp.Hq * inp.d * (2 if inp.dtype == "bf16" else 4)
    score_alg = key_b + q_bytes
    score_ms = score_prof["score_ms"]
    score_gbps = score_alg / (score_ms * 1e-3) / 1e9 if score_ms > 0 else None
    traffic = None if args.labels else counters_traffic()  # counters are of the exact stream
    log("measuring the plain streaming-read rate (read probe, 4 GiB)")
    peak_read = read_peak(torch, sd)

    rec = {
        "metric": METRIC,
        "value": inp.B / (ms_step * 1e-3),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if inp.dtype == "bf16" else "f32",
        "data": "synthetic (seeded; shapes and value structure of the workload)",
        "config": {"workload": synth.NAMES[args.workload], "batch": inp.B, "q_heads": inp.Hq,
                   "kv_heads": inp.Hkv, "head_dim": inp.d, "context": int(inp.ncap),
                   "sparsity": inp.ratio, "k": ks[0] if len(set(ks)) == 1 else "per sequence",
                   "layout": inp.layout, "group_shared": inp.group_shared,
                   **({"n_sink": inp.n_sink, "n_local": inp.n_local}
                      if inp.n_sink or inp.n_local else {}),
                   **({"fixed_k": args.fixed_k} if args.fixed_k is not None else {}),
                   **({"indexer": "8-channel bf16 labels"} if args.labels else {}),
                   **({"samples": args.samples} if args.samples else {})},
        "roofline": {
            "bound": "hbm",
            "kernel": "k_score_stream" + (" (label rows)" if args.labels else ""),
            "achieved": score_gbps,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": score_gbps / HBM_PEAK_GBPS if score_gbps else None,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": score_alg,
            "avg_launch_ms": score_ms,
            "measured_read_peak_GBps": peak_read,
            "frac_of_measured_read_peak": score_gbps / peak_read if score_gbps else None,
            "timing": "HIP events attached to every scoring dispatch (call's stream) over K "
                      "steps run right after the uninstrumented timed region",
        },
        "path": {
            "achieved_GBps": path_gbps,
            "frac_of_peak": path_gbps / HBM_PEAK_GBPS,
            "algorithmic_bytes": total_b,
            "key_stream_bytes": key_b,
            "value_gather_bytes": gather_b,
            "value_rows_gathered_per_head": sum(int(k) for k in ks) * inp.rows,
            "value_rows_union_per_kv_head": union_rows,
            "query_heads_per_s": inp.B * inp.Hq / (ms_step * 1e-3),
            "ms_per_step_events": ms_events,
            "ms_per_step_with_kernel_events": ms_timed_kernel,
            "stage_ms": {k_: round(prof[k_], 4) for k_ in
                         ("pilot_ms", "score_ms", "select_ms", "repair_ms", "attend_ms",
                          "total_ms")},
            "repaired_rows_last_step": prof["repaired_rows"],
        },
        "dense_baseline": dense,
        "calls_after_flush": calls,
    }
    # The target: the whole fused path at >= 70% of peak HBM bandwidth,
    # judged on the per-call median after a cache flush.
    if calls is not None and not args.labels and args.samples == 0:
        frac_flushed = total_b / (calls["median_ms"] * 1e-3) / 1e9 / HBM_PEAK_GBPS
        calls["path_frac_of_peak_at_median"] = frac_flushed
        rec["target"] = {"path_frac_required": 0.70,
                         "path_frac_back_to_back": path_gbps / HBM_PEAK_GBPS,
                         "path_frac_flushed_median": frac_flushed,
                         "met_flushed_median": frac_flushed >= 0.70,
                         "met_back_to_back": path_gbps / HBM_PEAK_GBPS >= 0.70}
    del q, cache, lens, out, idx, ws
    sd.set_workspace(None)
    torch.cuda.empty_cache()
    extras = [int(c) for c in args.extra_workloads.split(",") if c.strip()]
    extras = [c for c in extras if c != args.workload]
    if extras and not (args.labels or args.samples or args.sink or args.local or args.fixed_k
                       or args.ratio is not None):
        rec["extra_workloads"] = {f"workload{c}": extra_workload(args, c) for c in extras}
    if args.copy_mib > 0:
        n = args.copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        rec["copy_calibration_bytes"] = n
        del src, dst
    if args.cpu_sample > 0:
        log(f"timing the CPU oracle on {args.cpu_sample} sequences")
        rec["cpu_baseline"] = cpu_baseline(
            inp, args.cpu_sample, k_max, args.fixed_k, host_labels,
            draws=None if draws is None else draws.cpu().numpy().view(np.uint32))
    else:
        rec["cpu_baseline"] = None
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
