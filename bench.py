"""Benchmark of the hot path on one MI355X.

A step is one pass of the whole hot path over a resident batch: batched LPM
of every waiting request against the flattened cache tree (peek_lpm_batch),
then per-node demand and prefix-sharing clusters (peek_queue_signals). The
workload is the scale queue: 65536 prompts (60% RAG-shaped, 30% agentic,
10% random) against a cache tree of about one million nodes. The cache is
built once (not timed); prompts and cache are resident in HBM before the
timed region starts.

Prints one JSON line (rank 0). See --help for flags.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "LPM queries/sec + achieved HBM GB/s (% of peak), N=64K queue on 1 MI355X"
HBM_PEAK_GBS = 8000.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def block_algorithmic_bytes(lengths, block_h, B):
    """Bytes the hashed-block probe walk must move: the tokens of every full
    block it hashes (the hits and the first miss), one 8-byte table slot per
    probed block, the request's two offsets and its hit."""
    full = lengths // B
    probed = np.minimum(full, block_h // B + 1)
    return int((probed * B * 4).sum() + (probed * 8).sum() + len(lengths) * (16 + 4))


def walk_algorithmic_bytes(lengths, m, last, demand, exp):
    """Bytes the LPM walk must move: the prompt up to and including the first
    mismatch, the distinct cache edge tokens it compares, one 32-byte node
    record plus child probe per distinct node entered, offsets and outputs."""
    n = len(lengths)
    prompt = 4 * int(np.minimum(lengths, m + 1).sum())
    depth = exp["depth"].astype(np.int64)
    elen = exp["edge_len"].astype(np.int64)
    parent = exp["parent"].astype(np.int64)
    entered = demand > 0
    entered[0] = False
    # nodes passed through completely by at least one request
    last_cnt = np.bincount(last, minlength=len(depth))
    full = entered & (demand > last_cnt)
    compared = np.where(full, elen, 0)
    # nodes where some walk stopped: tokens compared up to the mismatch
    stop = last > 0
    lc = last[stop]
    dp = depth[parent[lc]]
    part = np.minimum(elen[lc], m[stop] - dp + 1)
    part_max = np.zeros(len(depth), dtype=np.int64)
    np.maximum.at(part_max, lc, part)
    compared = np.maximum(compared, np.where(entered, part_max, 0))
    edge_bytes = 4 * int(compared.sum())
    node_bytes = 32 * int(entered.sum())
    io_bytes = 8 * (n + 1) + 4 * 3 * n
    return prompt + edge_bytes + node_bytes + io_bytes, {
        "prompt_bytes": prompt, "edge_bytes": edge_bytes, "node_bytes": node_bytes, "io_bytes": io_bytes}


def measured_read_peak(torch) -> float:
    """GB/s of a plain streaming read of 4 GiB (libpeek_calib), best of 5."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2607_02525_amd", "libpeek_calib.so"))
    lib.peek_calib_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32,
                                           ctypes.c_void_p]
    nbytes = 4 << 30
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    times = []
    for _ in range(6):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        rc = lib.peek_calib_stream_read(ctypes.c_void_p(buf.data_ptr()), nbytes, ctypes.c_void_p(sink.data_ptr()),
                                        256 * 16, stream)
        b.record()
        torch.cuda.synchronize()
        assert rc == 0
        times.append(a.elapsed_time(b))
    del buf
    return nbytes / (min(times[1:]) / 1e3) / 1e9


WALK_SOURCES = ("peek_walk.hip", "peek_compare.h", "peek_internal.h")
WALK_COUNTERS = os.path.join(ROOT, "profiles", "k_lpm_walk_scale_counters.txt")


def walk_traffic(config: str, nodes: int, tokens: int):
    """HBM bytes per walk launch from the committed counter summary (FETCH_SIZE
    and WRITE_SIZE scaled by a plain-copy calibration), or None when the walk
    sources or the workload (cache nodes, queue tokens) changed since the
    counters were taken, or another config runs."""
    import hashlib
    if config != "scale" or not os.path.exists(WALK_COUNTERS):
        return None
    kv = {}
    for line in open(WALK_COUNTERS):
        if "=" in line and not line.startswith("#"):
            k, v = line.strip().split("=", 1)
            kv[k] = v
    h = hashlib.sha256()
    for f in WALK_SOURCES:
        with open(os.path.join(ROOT, "paper_2607_02525_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    if kv.get("source_sha256") != h.hexdigest():
        return None
    if kv.get("workload_nodes") != str(nodes) or kv.get("workload_tokens") != str(tokens):
        return None
    return int(kv["traffic_bytes_per_dispatch"])


def cpu_baseline(w, budget_s: float):
    """The oracle on one host core: LPM + demand + clusters over the whole
    queue, repeated for about budget_s seconds. Also returns the oracle's
    outputs of one pass (they fix the algorithmic byte counts)."""
    import oracle as O
    O.build(force=False)
    t0 = time.perf_counter()
    tree = O.cache_tree_of(w)
    ingest = time.perf_counter() - t0
    reps, total = 0, 0.0
    while total < budget_s or reps == 0:
        t = time.perf_counter()
        l = O.lpm(tree, w.tokens, w.offsets, w.block_size)
        d = O.demand(tree, l.last_node)
        c = O.clusters(w.tokens, w.offsets, w.threshold)
        total += time.perf_counter() - t
        reps += 1
    base = {"value": w.n * reps / total, "unit": "LPM queries/s", "cores": 1, "kind": "oracle",
            "sample": f"whole {w.name} queue ({w.n} requests): LPM + demand + clusters, single thread, "
                      f"{reps} passes in {total:.1f} s; cache-tree ingest {ingest:.1f} s not counted",
            "cpu": _cpu_model(), "host_logical_cpus": os.cpu_count()}
    return base, tree, (l, d, c)


def cpu_all_cores(w, tree, budget_s: float, threads: int):
    """The oracle's LPM + demand + clusters over the whole queue on `threads`
    host threads: the walk and the demand climb in request chunks (partial
    demands summed), the clusters per group of requests with the same first
    token (requests with different first tokens share nothing), groups dealt
    out largest first. The C calls release the interpreter lock."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle as O
    bounds = np.linspace(0, w.n, threads + 1).astype(np.int64)
    chunks = []
    for a, b in zip(bounds[:-1], bounds[1:]):
        off = w.offsets[a:b + 1]
        chunks.append((w.tokens[off[0]:off[-1]], off - off[0]))
    lens = np.diff(w.offsets)
    first = np.where(lens > 0, w.tokens[np.minimum(w.offsets[:-1], max(len(w.tokens) - 1, 0))], np.iinfo(np.int64).min)
    order = np.argsort(first, kind="stable")
    cuts = np.flatnonzero(np.diff(first[order])) + 1
    groups = sorted(np.split(order, cuts), key=len, reverse=True)
    group_queues = []
    for g in groups:
        g = np.sort(g)
        glen = lens[g]
        goff = np.zeros(len(g) + 1, np.int64)
        np.cumsum(glen, out=goff[1:])
        gtok = np.concatenate([w.tokens[w.offsets[i]:w.offsets[i + 1]] for i in g]) if len(g) > 1 else \
            w.tokens[w.offsets[g[0]]:w.offsets[g[0] + 1]]
        group_queues.append((gtok.astype(np.int32), goff))

    def walk_and_demand(cq):
        l = O.lpm(tree, cq[0], cq[1], w.block_size)
        return O.demand(tree, l.last_node)

    def cluster(gq):
        return O.clusters(gq[0], gq[1], w.threshold)

    reps, total, largest = 0, 0.0, 0.0
    with ThreadPoolExecutor(max_workers=threads) as ex:
        while total < budget_s or reps == 0:
            t = time.perf_counter()
            parts = list(ex.map(walk_and_demand, chunks))
            sum(parts)
            list(ex.map(cluster, group_queues))
            total += time.perf_counter() - t
            reps += 1
    return {"value": w.n * reps / total, "unit": "LPM queries/s", "cores": threads, "kind": "oracle",
            "sample": f"whole {w.name} queue ({w.n} requests): LPM + demand in {threads} request chunks, clusters "
                      f"in {len(groups)} first-token groups (largest {len(groups[0])} requests), {threads} threads, "
                      f"{reps} passes in {total:.1f} s",
            "host_logical_cpus": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)),
            "cpu": _cpu_model()}


def _cpu_model():
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def signals_algorithmic_bytes(lengths, share, m, n_nodes, passes):
    """The signals pass's bytes as the survey's byte accounting counts them:
    every prompt up to and including the token after its share (what a
    plain pending-tree build reads), 16 bytes per request per sort pass, 4
    of outputs, 16 per cache node (demand). Also the part of the prompt
    bytes the walk had already proven (up to the match length), which the
    pass here does not read again."""
    prompt = 4 * int(np.minimum(lengths, share + 1).sum())
    proven = 4 * int(np.minimum(np.minimum(lengths, share + 1), m).sum())
    n = len(lengths)
    parts = {"prompt_bytes": prompt, "sort_bytes": 16 * n * passes, "io_bytes": 4 * n,
             "node_bytes": 16 * n_nodes, "prompt_bytes_proven_by_the_walk": proven}
    return prompt + 16 * n * passes + 4 * n + 16 * n_nodes, parts


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="scale")
    ap.add_argument("--seed", type=int, default=42)
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB device-to-device copy (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: this hot path is built and measured on a single MI355X "
              "(multi-GPU sharding is described in the design notes, not built).", file=sys.stderr)
        sys.exit(2)

    import torch

    import peek_workloads as W
    import paper_2607_02525_amd as P
    from paper_2607_02525_amd import peek_cache_export
    from paper_2607_02525_amd.runner import HotPath

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    w = W.make(args.config, args.seed)
    log(f"workload {w.name} n={w.n} tokens={len(w.tokens)} generated in {time.perf_counter() - t0:.1f}s")
    t0 = time.perf_counter()
    if w.cache_tree is not None:
        hp = HotPath.from_description(*w.cache_tree)
    else:
        hp = HotPath.from_sequences(*w.cache_sequences)
    build_s = time.perf_counter() - t0
    stats = hp.cache.stats()
    log(f"cache built in {build_s:.1f}s: {stats}")
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        hp.step()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} done")

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        a, b, c = ev[i]
        a.record(stream)
        hp.lpm()
        b.record(stream)
        hp.signals()
        c.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    lpm_ms = np.array([e[0].elapsed_time(e[1]) for e in ev])
    sig_ms = np.array([e[1].elapsed_time(e[2]) for e in ev])
    ms_per_step = wall * 1e3 / args.steps
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step (lpm {lpm_ms.mean():.3f} ms, signals {sig_ms.mean():.3f} ms)")

    # the rest of cLPM's signal vector (score, section, has_sharing) on the
    # same queue: one peek_clpm_signals call replaces peek_queue_signals
    clpm_ms = []
    for i in range(max(3, args.steps // 2) + 1):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        hp.clpm(w.tau, w.theta)
        b.record(stream)
        torch.cuda.synchronize()
        if i > 0:
            clpm_ms.append(a.elapsed_time(b))
    log(f"cLPM signals (clusters + demand + score + section + has_sharing): {np.mean(clpm_ms):.3f} ms")
    # eviction ranking of the cached nodes from that demand (scores + victim order)
    evict_ms = []
    for i in range(4):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        hp.evict()
        b.record(stream)
        torch.cuda.synchronize()
        if i > 0:
            evict_ms.append(a.elapsed_time(b))
    log(f"eviction ranking of {hp.num_nodes} cached nodes: {np.mean(evict_ms):.3f} ms")

    # the hashed-block cache variant on the same tree and queue: table built
    # once on the host, then one probe walk per request
    t0 = time.perf_counter()
    table = hp.block_table(w.block_size)
    table_s = time.perf_counter() - t0
    block_ms = []
    for i in range(4):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        hp.block_lpm()
        b.record(stream)
        torch.cuda.synchronize()
        if i > 0:
            block_ms.append(a.elapsed_time(b))
    log(f"hashed-block LPM ({table.stats()['num_blocks']} stored blocks, table built in {table_s:.1f}s): "
        f"{np.mean(block_ms):.3f} ms")

    # PEEK-offline Phase 1 (D = 128) over the whole queue, and over its first
    # 5000 requests (the queue size the paper times its reorder at)
    def time_offline(fn, reps=4):
        ms = []
        for i in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            if i > 0:
                ms.append(a.elapsed_time(b))
        return float(np.mean(ms))

    offline_ms = time_offline(lambda: hp.offline(128))
    n5 = min(5000, w.n)
    sub_off = torch.from_numpy(np.ascontiguousarray(w.offsets[:n5 + 1] - w.offsets[0])).cuda()
    sub_tok = hp.d_tokens[int(w.offsets[0]):int(w.offsets[n5])]
    sub_perm = torch.empty(max(n5, 1), dtype=torch.int32, device="cuda")
    sub_ws = torch.empty(max(P.peek_offline_order_workspace(n5), 256), dtype=torch.uint8, device="cuda")
    offline5k_ms = time_offline(lambda: P.peek_offline_order(sub_tok, sub_off, 128, sub_perm, sub_ws))
    log(f"offline Phase 1 order (D = 128): {offline_ms:.3f} ms for {w.n} requests, {offline5k_ms:.3f} ms for {n5}")

    res = hp.results()
    block_bytes = block_algorithmic_bytes(w.lengths.astype(np.int64), res["block_h"].astype(np.int64),
                                          w.block_size)
    exp = peek_cache_export(hp.cache)
    b_alg, parts = walk_algorithmic_bytes(w.lengths.astype(np.int64), res["match_len"].astype(np.int64),
                                          res["last_node"].astype(np.int64), res["demand"].astype(np.int64), exp)
    lpm_avg_s = float(lpm_ms.mean()) / 1e3
    achieved = b_alg / lpm_avg_s / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": walk_traffic(args.config, hp.num_nodes, len(w.tokens)),
                "kernel": "k_lpm_walk", "algorithmic_bytes_per_launch": b_alg, "bytes_breakdown": parts,
                "bytes_from": "GPU outputs (no oracle run)",
                "avg_launch_ms": round(float(lpm_ms.mean()), 4), "min_launch_ms": round(float(lpm_ms.min()), 4)}

    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("calibration copy: 3 x 1 GiB device-to-device")
        del src, dst

    # achievable streaming-read bandwidth on this device (a plain 4 GiB read)
    read_peak = measured_read_peak(torch)
    roofline["measured_read_peak_gbs"] = round(read_peak, 1)
    roofline["frac_of_measured_read_peak"] = round(achieved / read_peak, 4)
    log(f"streaming read of 4 GiB: {read_peak:.0f} GB/s")

    cpu = cpu_all = None
    signals_roofline = None
    if not args.no_cpu_baseline:
        log("timing the oracle on the host for cpu_baseline")
        cpu, tree, (ol, od, oc) = cpu_baseline(w, args.cpu_budget)
        # the byte counts come from the oracle's outputs; the GPU's agree
        assert np.array_equal(ol.m, res["match_len"]) and np.array_equal(ol.last_node, res["last_node"])
        assert np.array_equal(od, res["demand"])
        b_alg, parts = walk_algorithmic_bytes(w.lengths.astype(np.int64), ol.m.astype(np.int64),
                                              ol.last_node.astype(np.int64), od.astype(np.int64), exp)
        roofline.update({"achieved": round(b_alg / lpm_avg_s / 1e9, 1),
                         "frac": round(b_alg / lpm_avg_s / 1e9 / HBM_PEAK_GBS, 4),
                         "algorithmic_bytes_per_launch": b_alg, "bytes_breakdown": parts,
                         "bytes_from": "oracle outputs"})
        # sort passes over the queue in one signals call: the first round's
        # merge sort (a tile pass over 512-element tiles, then merge passes)
        # and the sort of the second round's segments
        np2 = 512
        while np2 < w.n:
            np2 <<= 1
        tile = 1024 if np2 >= (1 << 19) else 512   # sorts of 512K elements and up use 1024-element tiles
        passes = 1 + int(np.log2(np2 // tile)) + 1
        sb, sparts = signals_algorithmic_bytes(w.lengths.astype(np.int64), oc.share.astype(np.int64),
                                               ol.m.astype(np.int64), hp.num_nodes, passes)
        sig_s = float(sig_ms.mean()) / 1e3
        signals_roofline = {"bound": "hbm", "achieved": round(sb / sig_s / 1e9, 1), "peak": HBM_PEAK_GBS,
                            "unit": "GB/s", "frac": round(sb / sig_s / 1e9 / HBM_PEAK_GBS, 4),
                            "call": "peek_queue_signals", "algorithmic_bytes_per_call": sb,
                            "bytes_breakdown": sparts, "sort_passes": passes,
                            "avg_call_ms": round(float(sig_ms.mean()), 4), "host_round_trips": 0}
        threads = max(1, min(16, len(os.sched_getaffinity(0))))
        cpu_all = cpu_all_cores(w, tree, args.cpu_budget / 2, threads)
        log(f"oracle LPM + demand + clusters on {threads} threads: {cpu_all['value']:.0f} queries/s "
            f"(host shows {os.cpu_count()} logical CPUs)")

    out = {
        "metric": METRIC,
        "value": round(w.n / (ms_per_step / 1e3), 1),
        "unit": "LPM queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.n} prompts ({len(w.tokens)} tokens), cache tree "
                               f"{stats['num_nodes']} nodes / {stats['num_edge_tokens']} edge tokens, "
                               f"block {w.block_size}, cluster threshold {w.threshold}, seed {w.seed}",
                   "queue": w.n, "parallelism": "single GPU"},
        "lpm_queries_per_s": round(w.n / lpm_avg_s, 1),
        "lpm_ms": round(float(lpm_ms.mean()), 4),
        "signals_ms": round(float(sig_ms.mean()), 4),
        "clpm_signals_ms": round(float(np.mean(clpm_ms)), 4),
        "evict_rank_ms": round(float(np.mean(evict_ms)), 4),
        # algorithmic bytes per cached node: demand 4, record 32, score 8, order 4
        "evict_rank_gbs": round(48 * hp.num_nodes / (float(np.mean(evict_ms)) / 1e3) / 1e9, 1),
        "block_lpm_ms": round(float(np.mean(block_ms)), 4),
        "block_lpm_gbs": round(block_bytes / (float(np.mean(block_ms)) / 1e3) / 1e9, 1),
        "block_table_build_s": round(table_s, 2),
        "offline_order_ms": round(offline_ms, 4),
        "offline_order_5000_ms": round(offline5k_ms, 4),
        "cache_build_s": round(build_s, 2),
        "roofline": roofline,
        "signals_roofline": signals_roofline,
        "cpu_baseline": cpu,
        "cpu_baseline_all_cores": cpu_all,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
