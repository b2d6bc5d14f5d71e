#!/usr/bin/env python3
"""Benchmark of the exact dense-retrieval hot path on one MI355X.

One step = one ``dresd_search`` call (sampled threshold passes, the main scan
over every key, merge and continuation gather) for one batch of queries,
cycling through the workload's query pool.  Inputs are resident in HBM before
the timed region starts.  Prints one JSON line.

Default workload: 1,048,576 keys x 4096 dims bf16 (a 7B model's hidden width),
continuations [N,10], B = 1 query per step, k = 10.  The default run also
measures, in the same JSON line under "secondary", the 33.5M x 128 f16
datastore at B = 1 and B = 128 (k = 100) and the 10M x 256 f16 datastore at
B = 256 (k = 32), each with its own roofline block, and under
"filtered_token_groups" the next-token-filtered search of the 33.5M-key
datastore grouped by first token at B = 1 beside the full filtered scan.  The
achievable read bandwidth of the device (a probe with the scans' access
pattern) is measured on the same run and each bandwidth is also given as a
fraction of it.  The
CPU-baseline leg times the oracle and checks query 0 of every measured
workload against it (outside the timed regions).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f16": 2500.0, "f32": 157.3}
CSRC = os.path.join(ROOT, "paper_2502_15572_amd", "csrc")
DEFAULT_WORKLOAD = "hidden1m_d4096_bf16"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


SCAN_UNIT = {"single_tile": "dresd_kernels.hip", "shared_key": "dresd_scan_mq.hip",
             "single_tile_grouped": "dresd_kernels.hip", "tiled": "dresd_scan_mq.hip"}
SCAN_KERNEL_NAME = {"single_tile": "dresd_scan_main", "shared_key": "dresd_scanmq_main",
                    "single_tile_grouped": "dresd_scan_main_shared", "tiled": "dresd_scantc_main"}


def kernel_hash(unit: str) -> str:
    """Hash of one kernel source file and every header it includes (a counter
    summary is valid only for the code it was taken on)."""
    seen, todo = [], [unit]
    while todo:
        f = todo.pop()
        if f in seen or not os.path.exists(os.path.join(CSRC, f)):
            continue
        seen.append(f)
        todo += re.findall(r'^#include "([^"]+)"', open(os.path.join(CSRC, f)).read(), re.M)
    h = hashlib.sha256()
    for f in sorted(seen):
        h.update(f.encode() + open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()[:16]


def read_traffic(workload: str, batch: int, scan_kernel: str):
    """HBM bytes per main-scan launch from the committed rocprofv3 counter
    summary, if it was taken on the current source of that scan kernel; else
    None."""
    path = os.path.join(ROOT, "profiles", "traffic_scan_%s_B%d.md" % (workload, batch))
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    m = re.search(r"^kernel_source_sha256_16:\s*(\S+)", txt, re.M)
    b = re.search(r"^hbm_bytes_per_launch:\s*([0-9.eE+]+)", txt, re.M)
    if not m or not b or m.group(1) != kernel_hash(SCAN_UNIT[scan_kernel]):
        return None
    return float(b.group(1))


def search_latency(run, steps: int):
    """p50 and p90 device time of one search (ms): events on the current
    stream around each of `steps` searches, in a loop of its own so that the
    timed region carries no per-search events."""
    import torch
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for i in range(steps):
        ev[i][0].record(stream)
        run(i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    per = sorted(a.elapsed_time(b) for a, b in ev)
    return statistics.median(per), per[min(len(per) - 1, int(0.9 * len(per)))]


def copy_calibration(nbytes: int):
    """A plain device copy of known size, to scale the HBM byte counters."""
    import torch
    n = nbytes // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 3}))


def cpu_baseline_leg(keys_dev, cont_dev, queries, k, device_result, budget_s=12.0, time_it=True,
                     next_tok=None):
    """The oracle (untuned) on this host's cores.  Checks the device's result
    for queries[0] against the oracle's exact top-k (rules R1-R7 of the
    parity tests; outside every timed region; with ``next_tok``, the
    next-token-filtered top-k for next_tok[0]) and, with ``time_it``, times
    single-query oracle searches over a bounded sample.  Returns
    (cpu_baseline dict or None, parity dict)."""
    import numpy as np
    import oracle
    from datagen import to_numpy_bits
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from parity import TOL, ParityError, check_query, check_query_filtered
    threads = len(os.sched_getaffinity(0))
    t0 = time.time()
    kb, dt = to_numpy_bits(keys_dev)
    cont = cont_dev.cpu().numpy()
    log("cpu_baseline: host copy of keys %.1fs" % (time.time() - t0))
    q = queries.cpu().numpy().astype(np.float32)
    nt0 = None if next_tok is None else int(next_tok[0])
    o_idx, o_score, _, o_next = oracle.topk(kb, dt, q[:1], k, cont, threads=threads,
                                            next_tok=None if nt0 is None else [nt0])
    g_idx, g_score, g_tok = (t[0].cpu().numpy() for t in device_result)
    parity = {"queries_checked": 1, "against": "oracle exact top-k (fp64 sums rounded once)"
              + ("" if nt0 is None else ", next-token filtered")}
    try:
        args = (g_idx, g_score, g_tok, o_idx[0], o_score[0], o_next[0],
                lambda rows: oracle.score_rows(kb, dt, q[0], rows), kb.shape[0], cont)
        rep = (check_query(*args, TOL[dt]) if nt0 is None
               else check_query_filtered(*args, nt0, TOL[dt]))
        parity.update({"verdict": "pass", "tol": TOL[dt], "exact_order": rep["exact_order"],
                       "max_abs_vs_exact": rep["max_abs_vs_exact"]})
    except ParityError as e:
        parity.update({"verdict": "FAIL", "tol": TOL[dt], "error": str(e)})
    base = None
    if time_it:
        done, t = 0, time.time()
        while time.time() - t < budget_s:
            b = done % q.shape[0]
            oracle.topk(kb, dt, q[b:b + 1], k, threads=threads)  # B = 1, as the metric
            done += 1
        el = time.time() - t
        base = {"value": done / el, "unit": "queries/s", "cores": threads, "kind": "oracle",
                "sample": "%d single-query searches over the full datastore (cycling the query "
                          "pool) in %.1f s, after one untimed search (the parity check of "
                          "query 0)" % (done, el)}
    del kb
    return base, parity


def bandwidth_probe(buf):
    """Achievable read bandwidth (GB/s): the library's probe over `buf` with
    the scans' access pattern, best over a few grid sizes."""
    import torch
    from paper_2502_15572_amd import bw_probe
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    best, per = 0.0, {}
    for wpc in (1, 2, 4, 8):
        gbps = bw_probe(buf, reps=10, workgroups=wpc * cus)
        per["%d_per_cu" % wpc] = gbps
        best = max(best, gbps)
    return best, per


def time_transform(args):
    """Time the query-side transform (z-score, projection, L2) of B rows."""
    import torch
    from datagen import WORKLOADS
    from paper_2502_15572_amd import transform
    w = WORKLOADS[args.workload]
    B, D, l = args.batch, args.transform, w.d
    g = torch.Generator(device="cuda").manual_seed(0)
    x = torch.randn(B, D, device="cuda", generator=g)
    mean = torch.randn(D, device="cuda", generator=g)
    var = torch.rand(D, device="cuda", generator=g) + 0.5
    W = torch.randn(D, l, device="cuda", generator=g) / D ** 0.5
    y = torch.empty(B, l, device="cuda")
    for _ in range(args.warmup):
        transform(x, mean, var, W, out=y)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for a, b in ev:
        a.record()
        transform(x, mean, var, W, out=y)
        b.record()
    torch.cuda.synchronize()
    per = sorted(a.elapsed_time(b) for a, b in ev)
    p50 = statistics.median(per)
    flops = 2.0 * B * D * l
    byts = 4.0 * (B * D + D * l + 2 * D + 2 * B * l)
    print(json.dumps({"transform": {"B": B, "D": D, "l": l, "p50_us": p50 * 1e3,
                                    "TFLOPs": flops / (p50 * 1e-3) / 1e12,
                                    "frac_fp32_mfma_peak": flops / (p50 * 1e-3) / 157.3e12,
                                    "GBps": byts / (p50 * 1e-3) / 1e9}}), flush=True)


def time_drafts(args):
    """Time draft assembly (Section 3.6) of B queries' k retrieved
    continuations into r EOS-padded drafts of `length` tokens.  Tokens are
    drawn from a 64-token vocabulary so repeated drafts and EOS are common."""
    import torch
    from datagen import WORKLOADS
    from paper_2502_15572_amd import pack_drafts
    w = WORKLOADS[args.workload]
    k = args.k or w.k
    B, L = args.batch, w.L
    r, length = min(args.drafts, k), L
    g = torch.Generator(device="cuda").manual_seed(0)
    tok = torch.randint(0, 64, (B, k, L), device="cuda", generator=g, dtype=torch.int32)
    drafts = torch.empty((B, r, length), dtype=torch.int32, device="cuda")
    count = torch.empty((B,), dtype=torch.int32, device="cuda")
    for _ in range(args.warmup):
        pack_drafts(tok, r, length, out=(drafts, count))
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for a, b in ev:
        a.record()
        pack_drafts(tok, r, length, out=(drafts, count))
        b.record()
    torch.cuda.synchronize()
    per = sorted(a.elapsed_time(b) for a, b in ev)
    p50 = statistics.median(per)
    byts = 4.0 * (B * k * L + B * r * length + B)
    print(json.dumps({"drafts": {"B": B, "k": k, "L": L, "r": r, "length": length,
                                 "p50_us": p50 * 1e3, "GBps": byts / (p50 * 1e-3) / 1e9,
                                 "mean_kept": float(count.float().mean())}}), flush=True)


def time_pipeline(args):
    """One decode step of retrieval (Algorithm 1 steps 4-8) on one stream:
    B hidden states of D fp32 dims -> transform (Eq. 1, a D x d projection
    standing in for the PCA basis, Eq. 2) -> next-token-filtered search of
    the workload's datastore (exact, or partitioned with --ivf P) -> draft
    assembly into 10 EOS-padded drafts.  Times the whole step."""
    import torch
    from datagen import WORKLOADS, generate
    from paper_2502_15572_amd import (Index, PartitionedIndex, kmeans_assign, pack_drafts,
                                      train_partitions, transform)
    w = WORKLOADS[args.workload]
    if args.n:
        w = w.scaled(args.n)
    k, B, D = args.k or w.k, args.batch, args.pipeline
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    g = generate(w, dev, with_queries=False)
    keys, cont = g["keys"], g["cont"]
    nprobe = args.nprobe[0]
    if args.ivf:
        pick = torch.randperm(w.N, generator=torch.Generator().manual_seed(1))
        sample = keys[pick[: min(w.N, args.train_rows_per_part * args.ivf)].to(dev)].contiguous()
        cents, _ = train_partitions(sample, args.ivf, iters=args.train_iters, seed=2)
        ix = PartitionedIndex(keys, cont, cents, kmeans_assign(keys, cents))
        search = lambda y, nt, out: ix.search(y, k, nprobe, out=out, next_tok=nt)
        kind = "partitioned P=%d nprobe=%d" % (args.ivf, nprobe)
    elif args.token_groups:
        ix = PartitionedIndex.by_first_token(keys, cont)
        search = lambda y, nt, out: ix.search_next_token(y, nt, k, out=out)
        kind = "exact, keys grouped by first token"
    else:
        ix = Index(keys, cont)
        search = lambda y, nt, out: ix.search(y, k, out=out, next_tok=nt)
        kind = "exact"
    torch.cuda.synchronize()
    log("index ready: %s, %s" % (w.name, kind))
    gen = torch.Generator(device="cuda").manual_seed(0)
    xs = torch.randn(64, B, D, device=dev, generator=gen)
    mean = torch.randn(D, device=dev, generator=gen)
    var = torch.rand(D, device=dev, generator=gen) + 0.5
    W = torch.randn(D, w.d, device=dev, generator=gen) / D ** 0.5
    # next token: the most frequent first token other than the EOS id (0)
    c0 = cont[: min(w.N, 1 << 20), 0]
    frequent = int(torch.mode(c0[c0 != 0]).values)
    nt = torch.full((B,), frequent, dtype=torch.int32, device=dev)
    y = torch.empty(B, w.d, device=dev)
    out = (torch.empty((B, k), dtype=torch.int64, device=dev),
           torch.empty((B, k), dtype=torch.float32, device=dev),
           torch.empty((B, k, w.L), dtype=torch.int32, device=dev))
    r = min(10, k)
    dout = (torch.empty((B, r, w.L), dtype=torch.int32, device=dev),
            torch.empty((B,), dtype=torch.int32, device=dev))

    def step(i):
        transform(xs[i % 64], mean, var, W, out=y)
        search(y, nt, out)
        pack_drafts(out[2], r, w.L, out=dout)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    p50, _ = search_latency(step, args.steps)
    print(json.dumps({"pipeline": {
        "workload": w.name, "N": w.N, "d": w.d, "D": D, "B": B, "k": k, "drafts": r,
        "search": kind,
        "steps_per_s": args.steps / el, "queries_per_s": args.steps * B / el,
        "p50_us": p50 * 1e3,
        "mean_drafts_kept": float(dout[1].float().mean())}}), flush=True)
    ix.close()


def time_partitioned(args):
    """Partitioned (inverted-file) search of the workload: spherical k-means
    on a seeded sample of the keys, every key assigned, then B-query searches
    at each nprobe.  Recall@k is measured against the exact search on the
    same queries; the scan's bandwidth counts the bytes of the probed
    partitions' keys (padding rows included)."""
    import torch
    from datagen import WORKLOADS, generate
    from paper_2502_15572_amd import Index, PartitionedIndex, kmeans_assign, train_partitions
    w = WORKLOADS[args.workload]
    if args.n:
        w = w.scaled(args.n)
    k = args.k or w.k
    B, P = args.batch, args.ivf
    w = w.with_pool(B)  # every batch holds B distinct queries
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t0 = time.time()
    g = generate(w, dev)
    keys, cont, pool = g["keys"], g["cont"], g["queries"]
    torch.cuda.synchronize()
    log("generated %s N=%d d=%d %s in %.1fs" % (w.name, w.N, w.d, w.dtype, time.time() - t0))
    t0 = time.time()
    ns = min(w.N, args.train_rows_per_part * P)
    pick = torch.randperm(w.N, generator=torch.Generator().manual_seed(1))[:ns].to(dev)
    sample = keys[pick].contiguous()
    cents, _ = train_partitions(sample, P, iters=args.train_iters, seed=2)
    del sample
    torch.cuda.synchronize()
    log("k-means on %d keys in %.1fs" % (ns, time.time() - t0))
    assign = kmeans_assign(keys, cents)
    torch.cuda.synchronize()
    train_s = time.time() - t0
    log("all keys assigned at %.1fs" % train_s)
    t0 = time.time()
    ivf = PartitionedIndex(keys, cont, cents, assign)
    build_s = time.time() - t0
    info = ivf.info()
    log("partitions: P=%d trained on %d rows in %.2fs, index built in %.2fs, %d tiles"
        % (P, ns, train_s, build_s, info["tiles"]))
    nb = max(1, pool.shape[0] // B)
    batches = [pool[i * B:(i + 1) * B].contiguous() for i in range(nb)]
    assert all(b.shape[0] == B for b in batches), "query pool smaller than the batch"
    nts = [None] * nb
    if args.filtered:  # as in the exact bench: the source row's first token
        c0 = cont[:, 0]
        frequent = int(torch.mode(c0[: min(w.N, 1 << 20)]).values)
        src = g["query_src"]
        nt = torch.where(src >= 0, c0[src.clamp(min=0)], torch.full_like(src, frequent))
        nt = nt.to(torch.int32)
        nts = [nt[i * B:(i + 1) * B].contiguous() for i in range(nb)]
    exact = Index(keys, cont)
    ref = [exact.search(b, k, tokens=False, next_tok=nts[i])[0] for i, b in enumerate(batches)]
    exact.close()
    # probed rows per query, from the same exact probing over the centroids
    cix = Index(cents, torch.arange(P, dtype=torch.int32, device=dev).view(P, 1))
    sizes = torch.bincount(assign.long(), minlength=P)
    padded = (sizes + 15) // 16 * 16
    for nprobe in args.nprobe:
        idx = torch.empty((B, k), dtype=torch.int64, device=dev)
        score = torch.empty((B, k), dtype=torch.float32, device=dev)
        tok = torch.empty((B, k, w.L), dtype=torch.int32, device=dev)
        out = (idx, score, tok)
        hits, total = 0, 0
        for i, b in enumerate(batches):
            ivf.search(b, k, nprobe, out=out, next_tok=nts[i])
            r = ref[i]
            for j in range(B):
                want = set(r[j].tolist()) - {-1}
                hits += len(set(idx[j].tolist()) & want)
                total += len(want)
        recall = hits / max(1, total)
        probe_rows, union_rows = 0, 0
        for b in batches:
            pr = cix.search(b, nprobe, tokens=False)[0]
            probe_rows += int(padded[pr].sum())
            union_rows += int(padded[torch.unique(pr)].sum())
        probe_rows /= nb * B
        union_rows /= nb
        log("nprobe %d: recall %.3f, timing ..." % (nprobe, recall))
        for i in range(args.warmup):
            ivf.search(batches[i % nb], k, nprobe, out=out, next_tok=nts[i % nb])
        torch.cuda.synchronize()
        ivf.profile(True)
        ivf.profile_read()
        t0 = time.perf_counter()
        for i in range(args.steps):
            ivf.search(batches[i % nb], k, nprobe, out=out, next_tok=nts[i % nb])
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        prof = ivf.profile_read()
        ivf.profile(False)
        p50, _ = search_latency(lambda i: ivf.search(batches[i % nb], k, nprobe, out=out,
                                                     next_tok=nts[i % nb]), args.steps)
        scan_ms = prof["scan_ms"] / max(1, prof["searches"])
        scan_bytes = probe_rows * B * w.d * w.elem_bytes
        print(json.dumps({
            "partitioned": {"workload": w.name, "N": w.N, "d": w.d, "key_dtype": w.dtype,
                            "B": B, "k": k, "P": P, "nprobe": nprobe,
                            "filtered": bool(args.filtered),
                            "queries_per_s": args.steps * B / el, "p50_latency_us": p50 * 1e3,
                            "recall_at_k": recall, "probed_rows_per_query": probe_rows,
                            "probed_fraction": probe_rows / w.N,
                            "batch_union_rows": union_rows,
                            "scan_kernel": "dresd_scan_parts", "scan_ms": scan_ms,
                            "scan_GBps": scan_bytes / (scan_ms * 1e-3) / 1e9,
                            "scan_hbm_frac": scan_bytes / (scan_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                            "train_rows": ns, "train_iters": args.train_iters,
                            "train_s": train_s, "index_build_s": build_s}}), flush=True)
    cix.close()
    ivf.close()


def time_token_groups(args):
    """Next-token-filtered search over keys grouped by the first token of
    their continuation (see token_groups_result); prints one JSON line."""
    import torch
    from datagen import WORKLOADS
    w = WORKLOADS[args.workload]
    if args.n:
        w = w.scaled(args.n)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    r = token_groups_result(w, args.batch, args.k or w.k, args, dev,
                            cpu=not args.no_cpu_baseline and not args.n)
    print(json.dumps({"token_groups": r}), flush=True)


def token_groups_result(w, B, k, args, dev, cpu=False):
    """Each query's next token is its source row's first token (as with
    --filtered), and each query scans only that token's group of keys.  The
    same batches also run through the full filtered scan, for the comparison
    and the agreement of the two results.  The scan bandwidth counts the
    bytes of the probed groups' keys (padding rows included).  With ``cpu``,
    query 0's grouped result is checked against the oracle's filtered top-k
    (outside the timed regions)."""
    import torch
    from datagen import generate
    from paper_2502_15572_amd import Index, PartitionedIndex
    w = w.with_pool(B)
    t0 = time.time()
    g = generate(w, dev)
    keys, cont, pool = g["keys"], g["cont"], g["queries"]
    torch.cuda.synchronize()
    log("generated %s N=%d d=%d %s in %.1fs" % (w.name, w.N, w.d, w.dtype, time.time() - t0))
    log("grouping the keys by first token ...")
    t0 = time.time()
    tix = PartitionedIndex.by_first_token(keys, cont)
    build_s = time.time() - t0
    info = tix.info()
    log("grouped by first token: %d groups, %d tiles, built in %.2fs"
        % (info["P"], info["tiles"], build_s))
    nb = max(1, pool.shape[0] // B)
    batches = [pool[i * B:(i + 1) * B].contiguous() for i in range(nb)]
    assert all(b.shape[0] == B for b in batches), "query pool smaller than the batch"
    c0 = cont[:, 0]
    frequent = int(torch.mode(c0[: min(w.N, 1 << 20)]).values)
    src = g["query_src"]
    nt = torch.where(src >= 0, c0[src.clamp(min=0)], torch.full_like(src, frequent))
    nt = nt.to(torch.int32)
    nts = [nt[i * B:(i + 1) * B].contiguous() for i in range(nb)]
    vals, counts = torch.unique(c0, return_counts=True)
    padded = (counts + 15) // 16 * 16
    pos = torch.searchsorted(vals, nt[: nb * B]).clamp(max=vals.numel() - 1)
    rows = torch.where(vals[pos] == nt[: nb * B], padded[pos], torch.zeros_like(padded[pos]))
    probe_rows = float(rows.float().mean())
    exact = Index(keys, cont)
    out_t = _search_buffers(B, k, w.L, dev)
    out_e = _search_buffers(B, k, w.L, dev)
    same, total = 0, 0
    for i, b in enumerate(batches):
        tix.search_next_token(b, nts[i], k, out=out_t)
        exact.search(b, k, out=out_e, next_tok=nts[i])
        same += int((out_t[0] == out_e[0]).all(dim=1).sum())
        total += B

    def timed(fn, prof_on, prof_read):
        for i in range(args.warmup):
            fn(i)
        torch.cuda.synchronize()
        prof_on(True)
        prof_read()
        t1 = time.perf_counter()
        for i in range(args.steps):
            fn(i)
        torch.cuda.synchronize()
        el = time.perf_counter() - t1
        prof = prof_read()
        prof_on(False)
        p50, _ = search_latency(fn, args.steps)
        return args.steps * B / el, p50, prof

    qps_t, p50_t, prof_t = timed(
        lambda i: tix.search_next_token(batches[i % nb], nts[i % nb], k, out=out_t),
        tix.profile, tix.profile_read)
    qps_e, p50_e, prof_e = timed(
        lambda i: exact.search(batches[i % nb], k, out=out_e, next_tok=nts[i % nb]),
        exact.profile, exact.profile_read)
    scan_ms = prof_t["scan_ms"] / max(1, prof_t["searches"])
    search_ms = prof_t["search_ms"] / max(1, prof_t["searches"])
    scan_bytes = probe_rows * B * w.d * w.elem_bytes
    res = {"workload": w.name, "N": w.N, "d": w.d, "key_dtype": w.dtype, "B": B, "k": k,
           "metric": "next-token-filtered retrieval over keys grouped by first token",
           "groups": info["P"], "queries_per_s": qps_t, "p50_latency_us": p50_t * 1e3,
           "scan_kernel": "dresd_scan_parts", "scan_ms": scan_ms, "search_ms": search_ms,
           "probed_rows_per_query": probe_rows, "probed_fraction": probe_rows / w.N,
           "scan_GBps": scan_bytes / (scan_ms * 1e-3) / 1e9,
           "scan_hbm_frac": scan_bytes / (scan_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
           "same_result_as_full_scan": same / max(1, total),
           "full_filtered_scan": {"queries_per_s": qps_e, "p50_latency_us": p50_e * 1e3,
                                  "search_ms": prof_e["search_ms"] / max(1, prof_e["searches"])},
           "speedup_p50": p50_e / p50_t, "index_build_s": build_s}
    exact.close()
    if cpu:
        checked = tuple(t.clone() for t in tix.search_next_token(batches[0], nts[0], k))
        torch.cuda.synchronize()
        log("oracle on the host (%s B=%d, grouped by first token) ..." % (w.name, B))
        _, res["parity"] = cpu_baseline_leg(keys, cont, batches[0], k, checked, time_it=False,
                                            next_tok=nts[0].cpu().tolist())
    tix.close()
    return res


def _search_buffers(B, k, L, dev):
    import torch
    return (torch.empty((B, k), dtype=torch.int64, device=dev),
            torch.empty((B, k), dtype=torch.float32, device=dev),
            torch.empty((B, k, L), dtype=torch.int32, device=dev))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None,
                    help="default: %s (and the secondary workloads)" % DEFAULT_WORKLOAD)
    ap.add_argument("--batch", type=int, default=None, help="default: 1")
    ap.add_argument("--k", type=int, default=0, help="default: the workload's k")
    ap.add_argument("--n", type=int, default=0, help="override N (reduced runs; not a bench line)")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the CPU-baseline leg (oracle timing and parity verdicts)")
    ap.add_argument("--no-secondary", action="store_true",
                    help="default run only: skip the secondary workloads")
    ap.add_argument("--bw-probe", action="store_true",
                    help="only measure the achievable read bandwidth (8 GiB buffer)")
    ap.add_argument("--filtered", action="store_true",
                    help="next-token-filtered search: each query's next token is the first "
                         "token of its source row's continuation (the most frequent first "
                         "token for queries without a source row)")
    ap.add_argument("--token-groups", action="store_true",
                    help="only time the next-token-filtered search over keys grouped by first "
                         "token (next tokens as with --filtered), beside the full filtered scan; "
                         "with --pipeline, the step's search")
    ap.add_argument("--transform", type=int, default=0, metavar="D",
                    help="only time the query-side transform: B rows of D fp32 dims projected "
                         "to the workload's d (Eq. 1, Section 3.3, Eq. 2)")
    ap.add_argument("--ivf", type=int, default=0, metavar="P",
                    help="only time the partitioned search with P k-means partitions")
    ap.add_argument("--nprobe", type=int, nargs="+", default=[16, 64, 256],
                    help="partitions probed per query (--ivf)")
    ap.add_argument("--train-rows-per-part", type=int, default=64,
                    help="k-means sample: this many keys per partition (--ivf)")
    ap.add_argument("--train-iters", type=int, default=10, help="k-means iterations (--ivf)")
    ap.add_argument("--pipeline", type=int, default=0, metavar="D",
                    help="only time one decode step of retrieval: B hidden states of D dims -> "
                         "transform -> filtered search (exact, or partitioned with --ivf) -> "
                         "10 drafts")
    ap.add_argument("--drafts", type=int, default=0, metavar="R",
                    help="only time draft assembly of the workload's k continuations into R "
                         "drafts (Section 3.6)")
    ap.add_argument("--copy-calibration", type=int, default=0,
                    help="only run a device copy of this many bytes (counter calibration)")
    args = ap.parse_args()
    # the secondary workloads belong to the default run only
    default_run = args.workload is None and args.batch is None
    args.workload = args.workload or DEFAULT_WORKLOAD
    args.batch = args.batch or 1

    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(--gpus %d requested)." % args.gpus, file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.bw_probe:
        import torch
        buf = torch.ones((8 << 30) // 4, dtype=torch.float32, device="cuda")
        best, per = bandwidth_probe(buf)
        print(json.dumps({"bw_probe": {"buffer_bytes": 8 << 30, "best_GBps": best,
                                       "frac_of_spec": best / HBM_PEAK_GBPS, "per_grid": per}}),
              flush=True)
        return
    if args.pipeline:
        time_pipeline(args)
        return
    if args.ivf:
        time_partitioned(args)
        return
    if args.token_groups:
        time_token_groups(args)
        return
    if args.drafts:
        time_drafts(args)
        return
    if args.transform:
        time_transform(args)
        return

    import torch
    from datagen import WORKLOADS

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    secondary = (default_run and not args.k and not args.n and not args.filtered
                 and not args.no_secondary)
    w = WORKLOADS[args.workload]
    if args.n:
        w = w.scaled(args.n)
    want_cpu = not args.no_cpu_baseline and not args.n
    res, peak = measure(w, args.batch, args.k or w.k, args, dev, probe=not args.n,
                        cpu=want_cpu, time_cpu=want_cpu and args.batch == 1 and not args.filtered)
    if secondary:
        res["secondary"] = []
        cache = {}
        for name, B in SECONDARY:
            ws = WORKLOADS[name]
            r, _ = measure(ws, B, ws.k, args, dev, cpu=want_cpu, time_cpu=False,
                           measured_peak=peak, cache=cache)
            res["secondary"].append(r)
        if cache.get("ix") is not None:
            cache["ix"].close()
        cache.clear()
        torch.cuda.empty_cache()
        wf = WORKLOADS[FILTERED_SECONDARY[0]]
        res["filtered_token_groups"] = token_groups_result(wf, FILTERED_SECONDARY[1], wf.k, args,
                                                           dev, cpu=want_cpu)
    print(json.dumps(res), flush=True)


# Secondary results of the default run: the datastore nearest to the paper's
# (33.5M keys, 128 dims, Zipf-sized clusters) at one query per step and at a
# 128-query batch, and the 10M x 256 datastore at 256 queries (the matrix-core
# regime).
SECONDARY = [("zipf33m_d128_f16", 1), ("zipf33m_d128_f16", 128), ("hidden1m_d4096_bf16", 64),
             ("batch10m_d256_f16", 256)]
# and the next-token-filtered search over the same 33.5M-key datastore grouped
# by first token, at one query per step, beside the full filtered scan
FILTERED_SECONDARY = ("zipf33m_d128_f16", 1)


def measure(w, B, k, args, dev, probe=False, cpu=False, time_cpu=False, measured_peak=None,
            cache=None):
    """Time `args.steps` searches of B queries on workload w (after
    `args.warmup`), with the library's per-kernel events for the main scan
    and the whole search.  Returns (result dict, measured read peak GB/s)."""
    import torch
    from datagen import generate
    from paper_2502_15572_amd import Index

    w = w.with_pool(B)  # every batch holds B distinct queries
    if cache is not None and cache.get("name") == (w.name, w.pool):
        g, ix, build_s = cache["g"], cache["ix"], cache["build_s"]
    else:
        if cache is not None and cache.get("ix") is not None:
            cache["ix"].close()
            cache.clear()
            torch.cuda.empty_cache()
        t0 = time.time()
        g = generate(w, dev)
        torch.cuda.synchronize()
        log("generated %s N=%d d=%d %s in %.1fs" % (w.name, w.N, w.d, w.dtype, time.time() - t0))
        t0 = time.time()
        ix = Index(g["keys"], g["cont"])
        build_s = time.time() - t0
        log("index built in %.2fs" % build_s)
        if cache is not None:
            cache.update(name=(w.name, w.pool), g=g, ix=ix, build_s=build_s)
    pool = g["queries"]
    nb = max(1, pool.shape[0] // B)
    batches = [pool[(i % nb) * B:(i % nb) * B + B].contiguous() for i in range(nb)]
    assert all(b.shape[0] == B for b in batches), "query pool smaller than the batch"
    tok_batches = [None] * nb
    if args.filtered:
        c0 = g["cont"][:, 0]
        frequent = int(torch.mode(c0[: min(w.N, 1 << 20)]).values)
        src = g["query_src"]
        nt = torch.where(src >= 0, c0[src.clamp(min=0)], torch.full_like(src, frequent))
        nt = nt.to(torch.int32)
        tok_batches = [nt[(i % nb) * B:(i % nb) * B + B].contiguous() for i in range(nb)]
    idx = torch.empty((B, k), dtype=torch.int64, device=dev)
    score = torch.empty((B, k), dtype=torch.float32, device=dev)
    tok = torch.empty((B, k, w.L), dtype=torch.int32, device=dev)
    out = (idx, score, tok)

    for i in range(args.warmup):
        ix.search(batches[i % nb], k, out=out, next_tok=tok_batches[i % nb])
    torch.cuda.synchronize()

    # Timed region: K back-to-back searches; the library times its main scan
    # kernel and each whole search with events tied to kernels' dispatches.
    ix.profile(True)
    ix.profile_read()  # clear
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ix.search(batches[i % nb], k, out=out, next_tok=tok_batches[i % nb])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = ix.profile_read()
    ix.profile(False)
    p50, p90 = search_latency(lambda i: ix.search(batches[i % nb], k, out=out,
                                                  next_tok=tok_batches[i % nb]), args.steps)
    # the result that the CPU-baseline leg checks: the first batch
    checked = tuple(t.clone() for t in ix.search(batches[0], k, next_tok=tok_batches[0]))
    torch.cuda.synchronize()

    peak = measured_peak
    probe_detail = None
    if probe:
        peak, probe_detail = bandwidth_probe(g["keys"])
        log("bandwidth probe: %.0f GB/s" % peak)

    s = w.elem_bytes
    scan_bytes = w.N * w.d * s + B * w.d * 4           # keys once + queries
    if args.filtered:
        scan_bytes += w.N * 4 + B * 4                  # first-token column + next tokens
    search_bytes = scan_bytes + B * k * (8 + 4 + 4 * w.L)
    scan_ms = prof["scan_ms"] / max(1, prof["searches"])
    search_ms = prof["search_ms"] / max(1, prof["searches"])
    achieved = scan_bytes / (scan_ms * 1e-3) / 1e9
    flops = 2.0 * w.N * w.d * B
    plan = ix.plan(B, k)
    kname = SCAN_KERNEL_NAME[plan["scan_kernel"]]
    # The scan's floor is the larger of its HBM time and its matrix-core time.
    mfma_peak = MFMA_PEAK_TFLOPS[w.dtype] * 1e12
    mfma_bound = flops / mfma_peak > scan_bytes / (HBM_PEAK_GBPS * 1e9)
    traffic = read_traffic(w.name, B, plan["scan_kernel"]) if not args.n else None
    search_gbps = search_bytes / (search_ms * 1e-3) / 1e9

    res = {
        "metric": "retrieval queries/s + p50 latency at B=1; achieved HBM GB/s vs peak",
        "value": args.steps * B / elapsed,
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "N": w.N, "d": w.d, "key_dtype": w.dtype, "B": B, "k": k,
                   "filtered": bool(args.filtered),
                   "L": w.L, "query_pool": int(pool.shape[0]),
                   "sample_passes": plan["sample_passes"], "scan_waves": plan["scan_waves"],
                   "scan_kernel": plan["scan_kernel"], "scan_launches": plan["launches"]},
        "p50_latency_us": p50 * 1e3,
        "p90_latency_us": p90 * 1e3,
        "search_hbm_GBps_at_p50": search_bytes / (p50 * 1e-3) / 1e9,
        "index_build_s": build_s,
        "roofline": {
            "bound": "mfma" if mfma_bound else "hbm",
            "kernel": kname,
            "achieved": (flops / (scan_ms * 1e-3) / 1e12) if mfma_bound else achieved,
            "peak": MFMA_PEAK_TFLOPS[w.dtype] if mfma_bound else HBM_PEAK_GBPS,
            "unit": "TFLOP/s" if mfma_bound else "GB/s",
            "frac": (flops / (scan_ms * 1e-3) / mfma_peak) if mfma_bound
                    else achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            # a batch that takes several launches (each a pass over the keys
            # for its part of the batch) counts the keys once: bytes, flops
            # and time are those of the whole batch's main scan
            "algorithmic_bytes_per_launch": scan_bytes,
            "algorithmic_flops_per_launch": flops,
            "avg_launch_ms": scan_ms,
            "launches": plan["launches"],
            "hbm_GBps": achieved,
            "hbm_frac": achieved / HBM_PEAK_GBPS,
            "hbm_frac_of_measured_peak": (achieved / peak) if peak else None,
            "mfma_util": flops / (scan_ms * 1e-3) / mfma_peak,
            # the whole search (sampled passes, main scan, merges, gather)
            "search_ms": search_ms,
            "search_hbm_GBps": search_gbps,
            "search_hbm_frac": search_gbps / HBM_PEAK_GBPS,
        },
    }
    if probe:
        res["measured_read_peak"] = {"GBps": peak, "frac_of_spec": peak / HBM_PEAK_GBPS,
                                     "kernel": "dresd_bw_read", "buffer_bytes":
                                     g["keys"].numel() * g["keys"].element_size(),
                                     "per_grid": probe_detail}
    if cpu:
        log("oracle on the host (%s B=%d) ..." % (w.name, B))
        # query 0 of the checked batch is pool[0]; the timing cycles the pool
        base, parity = cpu_baseline_leg(g["keys"], g["cont"], pool, k, checked,
                                        time_it=time_cpu)
        res["parity"] = parity
        if base is not None:
            res["cpu_baseline"] = base
    if cache is None:
        ix.close()
    return res, peak


if __name__ == "__main__":
    main()
