#!/usr/bin/env python3
"""Benchmark of the HUGE training step on one MI355X.

One "step" is one synchronous SGD step of skip-gram negative sampling over a
batch of (source_id, destination_id, co_counts) triples: sampling, grouping,
gather, loss, update.  Default workload: the 100M-node SBM (two 1e8 x 128
fp32 tables, 102.4 GB resident; 5 uniform negatives; 262,144 positives per
step), inputs pre-staged in HBM before the timed region.

Prints one JSON line with the throughput (positives per second), the
roofline of the dominant kernel (the fused gather/loss/update kernel, timed
with HIP events inside the timed steps on the stream it runs on), and the CPU
oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "positive (src,dst) pairs/sec per train step; achieved HBM GB/s vs peak"
HBM_PEAK_GBPS = 8000.0
FP16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 matrix peak
KERNEL = "k_fused_step"
COUNTERS_FILES = {  # committed rocprofv3 HBM counters of the fused kernel, per table type
    "f32": os.path.join(ROOT, "profiles", "fused_step_sbm100m_counters.txt"),
    "bf16": os.path.join(ROOT, "profiles", "fused_step_sbm100m_bf16_counters.txt"),
}
KERNEL_SOURCES = ["paper_2307_14490_amd/csrc/device.hpp", "paper_2307_14490_amd/csrc/k_step.hip"]
KERNEL_END = "// Lanes per row of the fused step and the probe."  # the fused kernel's source ends here
PROFILE_EVERY = 4  # timed steps whose fused kernel is bracketed by HIP events


def kernel_source_hash() -> str:
    """Hash of the fused kernel's source: device.hpp and k_step.hip up to the
    end of k_fused_step (the counters stay valid while neither changes)."""
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            text = f.read()
        if p.endswith("k_step.hip"):
            text = text[:text.index(KERNEL_END.encode())]
        h.update(text)
    return h.hexdigest()[:16]


def read_traffic(workload: str, dtype: str = "f32"):
    """HBM bytes per launch of the fused kernel from committed rocprofv3
    counters, if they were taken on the current kernel source."""
    path = COUNTERS_FILES.get(dtype)
    if workload != "sbm100m" or path is None or not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_hash") != kernel_source_hash():
        return None
    try:
        return float(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    """The host CPU's model name (first "model name" line of /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


# Steps of the CPU oracle per workload: a whole epoch of the tiny workload,
# the first 50 steps of the medium one, the first 5 of the large ones (all
# within the time budget).
CPU_STEPS = {"tiny": None, "medium": 50}
CPU_STEPS_DEFAULT = 5


def cpu_baseline(wl, seed, budget_s=30.0):
    """The CPU oracle on a bounded sample of the same workload, single
    threaded and pinned to one core of the calling thread's affinity set.

    Each step is the oracle's own work, timed call by call: its negative
    draws, the initial values of the rows the batch touches, and the double
    precision step (C code).  The numpy glue between those calls (the
    distinct row ids and the relabelling to them) is timed apart and not in
    the rate."""
    import numpy as np
    from oracle import oracle as orc
    cfg = wl.cfg
    thr = alias = None
    if cfg.neg_kind == "alias":
        thr, alias = orc.build_alias(wl.weights)
    a = float(np.float32(cfg.init_half_width))
    steps = CPU_STEPS.get(cfg.name, CPU_STEPS_DEFAULT)
    batch = wl.batch
    if steps is None:  # the epoch's corpus in batches
        corpus = wl.epoch()
        steps = -(-corpus[0].size // cfg.batch)

        def batch(b):
            return tuple(x[b * cfg.batch:(b + 1) * cfg.batch] for x in corpus)
    allowed = sorted(os.sched_getaffinity(0))
    core = allowed[0]
    os.sched_setaffinity(0, {core})
    t_oracle = t_glue = 0.0
    done = b = 0
    try:
        while b < steps and (t_oracle + t_glue < budget_s or b == 0):
            src, dst, cc = batch(b)
            first = b * cfg.batch
            t0 = time.perf_counter()
            neg = orc.sample_negatives(seed, first, src.size, cfg.num_neg, cfg.num_nodes, thr,
                                       alias)
            t1 = time.perf_counter()
            rows_S = np.unique(src.astype(np.int64))
            rows_T = np.unique(np.concatenate([dst.astype(np.int64),
                                               neg.reshape(-1).astype(np.int64)]))
            t2 = time.perf_counter()
            S = orc.init_rows(seed, 0, rows_S, cfg.dim, a)
            T = orc.init_rows(seed, 1, rows_T, cfg.dim, a)
            t3 = time.perf_counter()
            src_c = np.searchsorted(rows_S, src).astype(np.int32)
            dst_c = np.searchsorted(rows_T, dst).astype(np.int32)
            neg_c = np.searchsorted(rows_T, neg.reshape(-1)).astype(np.int32).reshape(
                src.size, cfg.num_neg)
            t4 = time.perf_counter()
            orc.step_dense(S, T, src_c, dst_c, cc, neg_c, cfg.lr)
            t5 = time.perf_counter()
            t_oracle += (t1 - t0) + (t3 - t2) + (t5 - t4)
            t_glue += (t2 - t1) + (t4 - t3)
            done += src.size
            b += 1
    finally:
        os.sched_setaffinity(0, set(allowed))
    return {
        "value": done / t_oracle,
        "unit": "positives/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"the first {b} step(s) of the {cfg.name} workload ({cfg.batch} positives "
                  f"each), each from initial values: negative draws, initial values of the "
                  f"touched rows and the double-precision step, {t_oracle:.1f} s; "
                  f"numpy glue (distinct ids, relabelling) {t_glue:.1f} s more, not in the rate",
        "pinned_core": core,
        "cpu_model": cpu_model(),
        "cores_total": os.cpu_count(),
        "cores_allowed": len(allowed),
        "glue_s": t_glue,
    }


def bench_producer(args):
    """The random-walk sampler on the exact SBM graph of a workload (default
    the 1M-node medium one) with the paper's sampling parameters (Table 2:
    128 walks of 3 steps per node; pairs of the seed with each visited node,
    their distance histograms): all seeds in chunks, timed with HIP events."""
    import numpy as np
    import torch

    import paper_2307_14490_amd as P
    from synth import make_workload

    def log(*a):
        print(*a, file=sys.stderr, flush=True)

    wl = make_workload(args.workload, args.seed)
    if wl.csr is None:
        raise SystemExit(f"--producer needs a workload with an exact graph (tiny, medium)")
    off, nbr = wl.csr
    N = wl.cfg.num_nodes
    gamma, steps, window = 128, 3, 3
    chunk = 65536
    doff = torch.from_numpy(np.asarray(off, np.int64)).cuda()
    dnbr = torch.from_numpy(np.asarray(nbr, np.int32)).cuda()
    log(f"[bench] graph: {N} nodes, {nbr.size} directed edges")
    cap = chunk * gamma * window
    cfg = P.walk_config(N, gamma, steps, window, True, args.seed)
    L = P.load()
    import ctypes
    ws_bytes = L.huge_walk_workspace_bytes(ctypes.byref(cfg), chunk)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    outs = [torch.empty(cap, dtype=torch.int32, device="cuda") for _ in range(3)]
    hist = torch.empty((cap, window), dtype=torch.int32, device="cuda")
    counts = torch.zeros(max(1, (N + chunk - 1) // chunk), dtype=torch.int64, device="cuda")
    status = torch.zeros(counts.numel(), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    def run_all():
        for c, s0 in enumerate(range(0, N, chunk)):
            ns = min(chunk, N - s0)
            rc = L.huge_sample_walks(ctypes.byref(cfg), doff.data_ptr(), dnbr.data_ptr(),
                                     dnbr.numel(), s0, ns, outs[0].data_ptr(),
                                     outs[1].data_ptr(), outs[2].data_ptr(), hist.data_ptr(),
                                     cap, counts[c:c + 1].data_ptr(),
                                     status[c:c + 1].data_ptr(), ws.data_ptr(), ws_bytes,
                                     ctypes.c_void_p(stream.cuda_stream))
            if rc != 0:
                raise P.HugeError(rc, "huge_sample_walks")

    run_all()  # warm-up
    torch.cuda.synchronize()
    if int(status.abs().max().item()) != 0:
        raise RuntimeError("the sampler reported an error")
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    reps = max(1, args.steps // 100)
    ev0.record(stream)
    for _ in range(reps):
        run_all()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / reps
    triples = int(counts.sum().item())
    walk_steps = N * gamma * steps
    value = triples / (ms * 1e-3)
    log(f"[bench] {triples} triples from {N} seeds in {ms:.2f} ms")
    # Algorithmic bytes: per walk step two offsets and one neighbour (20 B),
    # taken twice (counting pass and writing pass), plus the triples written
    # (src, dst, cc and a 3-entry histogram: 24 B each).
    alg_bytes = 2 * 20.0 * walk_steps + 24.0 * triples
    achieved = alg_bytes / (ms * 1e-3) / 1e9
    out = {
        "metric": "co-occurrence triples/sec (random-walk sampler)",
        "value": value,
        "unit": "triples/s",
        "n_gpus": 1,
        "steps": reps,
        "warmup": 1,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": f"{wl.cfg.name} graph, sampler", "num_nodes": N,
                   "edges": int(nbr.size), "walks_per_node": gamma, "walk_steps": steps,
                   "window": window, "pairs": "seed", "seeds_per_call": chunk},
        "roofline": {"kernel": "k_walk", "bound": "hbm", "achieved": achieved,
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": None,
                     "note": "dependent random 4-16 B reads: latency-bound, not bandwidth-bound"},
        "walk_steps_per_s": walk_steps / (ms * 1e-3),
    }
    if not args.no_cpu:
        from oracle import oracle as orc
        t0 = time.perf_counter()
        done = 0
        n_seeds = 0
        while time.perf_counter() - t0 < args.cpu_budget and n_seeds < N:
            r = orc.sample_walks(off, nbr, N, gamma, steps, window, True, args.seed,
                                 first_seed=n_seeds, num_seeds=min(2000, N - n_seeds))
            done += r[0].size
            n_seeds += min(2000, N - n_seeds)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": done / dt, "unit": "triples/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{n_seeds} seeds of the same graph and parameters, "
                                         f"{dt:.1f} s single-threaded"}
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


def bench_eval(args):
    """Unsupervised evaluation of embeddings (Sec. 4): on the medium exact SBM
    (1M nodes, trained for eight epochs of GPU-sampled walk triples) the whole
    evaluation -- 1M
    edge and 1M non-edge pairs, their distances, SNR and percentiles, the 10
    nearest rows of 100 sampled nodes and recall@10 -- each stage timed with
    HIP events; then the 100-query nearest-row search over the SBM-100M
    table (1e8 x 128 fp32), the dense contraction of the evaluation, timed
    against the fp32 matrix-core peak."""
    import numpy as np
    import torch

    import paper_2307_14490_amd as P
    from synth import make_workload, relabel

    def log(*a):
        print(*a, file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    def medium_evaluation():
        """The whole evaluation on the medium table, trained from GPU-sampled
        walks; returns its figures."""
        wl = make_workload("medium", args.seed)
        cfg = wl.cfg
        N, D = cfg.num_nodes, cfg.dim
        off0, nbr0 = wl.csr
        a = relabel(np.repeat(np.arange(N), np.diff(off0)), N, wl.perm)
        b = relabel(np.asarray(nbr0, np.int64), N, wl.perm)
        order = np.lexsort((b, a))
        a, b = a[order], b[order]
        off = np.zeros(N + 1, np.int64)
        np.add.at(off, a + 1, 1)
        off = np.cumsum(off)
        doff = torch.from_numpy(off).cuda()
        dnbr = torch.from_numpy(b.astype(np.int32)).cuda()
        tr = P.Trainer(N, D, cfg.num_neg, cfg.batch, seed=args.seed,
                       alias_weights=wl.weights if cfg.neg_kind == "alias" else None)
        # epochs of triples from the GPU walk sampler (a walk of the workload's
        # length and window from every node, new walks each epoch), shuffled on
        # the device
        epochs = 8
        train_steps = 0
        pos = 0
        g = torch.Generator(device="cuda")
        g.manual_seed(args.seed)
        for ep in range(epochs):
            ts, td, tc, _ = P.sample_walks(doff, dnbr, N, 1, cfg.walk_steps, cfg.window, False,
                                           args.seed + ep, with_hist=False)
            perm = torch.randperm(ts.numel(), device="cuda", generator=g)
            ts, td, tc = ts[perm].contiguous(), td[perm].contiguous(), tc[perm].contiguous()
            for i0 in range(0, ts.numel(), cfg.batch):
                i1 = min(i0 + cfg.batch, ts.numel())
                tr.step_no_loss(ts[i0:i1], td[i0:i1], tc[i0:i1], pos, cfg.lr)
                pos += i1 - i0
                train_steps += 1
            del ts, td, tc, perm
        if tr.check() != 0:
            raise RuntimeError("device reported an error while training")
        log(f"[bench] medium: {N} nodes, {b.size} directed edges, trained {epochs} epochs of "
            f"walk triples ({pos} positives, {train_steps} steps)")
        ne = nn = 1_000_000
        nq, k = 100, 10
        ev = P.Evaluator(N, D, ne + nn, k=k)
        qs = torch.from_numpy(np.random.default_rng(args.seed).choice(N, nq, replace=False)
                              .astype(np.int32)).cuda()
        reps = 5
        t_pairs = timed(lambda: ev.pairs(doff, dnbr, N, args.seed, ne, nn), reps)
        u, v = ev.pairs(doff, dnbr, N, args.seed, ne, nn)
        t_dist = timed(lambda: ev.distances(tr.S, u, v), reps)
        dist = ev.distances(tr.S, u, v)
        quant = list(range(0, 101, 10))
        t_sum = timed(lambda: ev.summary(dist, ne, nn, quant), reps)
        summ = ev.summary(dist, ne, nn, quant)
        t_knn_m = timed(lambda: ev.knn(tr.S, qs, k), reps)
        ids, _ = ev.knn(tr.S, qs, k)
        t_rec = timed(lambda: ev.recall(doff, dnbr, N, qs, ids), reps)
        rec = ev.recall(doff, dnbr, N, qs, ids)
        medium = {"num_nodes": N, "dim": D, "edges": int(b.size), "trained_steps": train_steps,
                  "trained_positives": pos,
                  "pairs": ne + nn, "queries": nq, "k": k,
                  "ms": {"pairs": t_pairs, "distances": t_dist, "summary": t_sum, "knn": t_knn_m,
                         "recall": t_rec},
                  "snr": summ["snr"], "mean_edge": summ["mean_edge"],
                  "mean_non": summ["mean_non"], "pct_edge": summ["pct_edge"],
                  "pct_non": summ["pct_non"], "percentiles": quant,
                  "recall_at_10_mean": float(rec.mean().item()),
                  "distances_GBps": (ne + nn) * 2 * 4 * D / (t_dist * 1e-3) / 1e9}
        log(f"[bench] medium evaluation: SNR {summ['snr']:.3f}, recall@10 "
            f"{medium['recall_at_10_mean']:.3f}; ms {medium['ms']}")
        del tr, ev, u, v, dist
        torch.cuda.empty_cache()
        return medium

    # ---- medium: the whole evaluation on a trained table (skipped with
    # --knn-only, which times the large search alone)
    nq, k = 100, 10
    medium = None if args.knn_only else medium_evaluation()

    # ---- SBM-100M table: the 100-query nearest-row search
    big = make_workload("sbm100m", args.seed).cfg
    NB, DB = big.num_nodes, big.dim
    trb = P.Trainer(NB, DB, big.num_neg, 1024, seed=args.seed)
    evb = P.Evaluator(NB, DB, 8, k=k)
    qb = torch.from_numpy(np.random.default_rng(args.seed + 1).choice(NB, nq, replace=False)
                          .astype(np.int32)).cuda()
    breps = max(2, args.steps // 40)
    t_knn = timed(lambda: evb.knn(trb.S, qb, k), breps)
    idsb, db = evb.knn(trb.S, qb, k)
    # same-box context: the library's own reduction over the same table (one
    # plain read, no search); not a ceiling (the search reads faster)
    t_read = timed(lambda: trb.S.sum(), breps)
    read_gbps = NB * DB * 4 / (t_read * 1e-3) / 1e9
    flops = 2.0 * NB * DB * nq
    achieved = flops / (t_knn * 1e-3) / 1e12
    qpad = 128
    # the table read once, and the fp16 matrix work of the screen (one hi.hi
    # product per dimension, 128 query slots)
    table_gbps = NB * DB * 4 / (t_knn * 1e-3) / 1e9
    fp16_ms = 2 * NB * DB * qpad / FP16_PEAK_TFLOPS / 1e9
    log(f"[bench] knn over {NB} x {DB}: {t_knn:.2f} ms, {achieved:.1f} TFLOP/s algorithmic, "
        f"table read at {table_gbps:.0f} GB/s (torch.sum over the table: {t_read:.2f} ms, "
        f"{read_gbps:.0f} GB/s)")
    # sampled check of the result: the returned rows' exact distances, and no
    # row of a random sample nearer than the k-th (property at any size)
    rng = np.random.default_rng(7)
    samp = np.sort(rng.choice(NB, 200_000, replace=False))
    Sq = trb.S[qb.long()].double().cpu().numpy()
    Ss = trb.S[torch.from_numpy(samp).cuda()].double().cpu().numpy()
    qn = Sq / np.linalg.norm(Sq, axis=1, keepdims=True)
    sn = Ss / np.linalg.norm(Ss, axis=1, keepdims=True)
    d2s = np.maximum(2.0 - 2.0 * qn @ sn.T, 0.0)
    kth = db[:, k - 1].double().cpu().numpy() ** 2
    got = idsb.cpu().numpy()
    returned = np.zeros(d2s.shape, bool)       # sampled rows the search returned
    for qi in range(nq):
        returned[qi] = np.isin(samp, got[qi])
    ok = np.all((d2s >= kth[:, None] - 4 * DB * 2.0 ** -24 - 1e-6) | returned |
                (samp[None, :] == qb.cpu().numpy()[:, None]))
    if not ok:
        raise RuntimeError("a sampled row is nearer than the returned k-th row")
    out = {
        "metric": "query-row distances/sec (100-query nearest-row search, Sec. 4 recall)",
        "value": NB * nq / (t_knn * 1e-3),
        "unit": "distances/s",
        "n_gpus": 1,
        "steps": breps,
        "warmup": 1,
        "ms_per_step": t_knn,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "SBM-100M table (1e8 x 128 fp32, initial values), 100 queries, "
                               "k = 10", "num_rows": NB, "dim": DB, "queries": nq, "k": k},
        "roofline": {"kernel": "k_knn_scan<4, true>", "bound": "hbm", "achieved": table_gbps,
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": table_gbps / HBM_PEAK_GBPS,
                     "traffic": None,
                     "note": f"the whole search (three sample scans over 3.2% of the tiles, the "
                             f"full scan, four selections) against one read of the "
                             f"{NB * DB * 4 / 1e9:.1f} GB table: "
                             f"{NB * DB * 4 / HBM_PEAK_GBPS / 1e6:.1f} ms at the HBM peak; the "
                             f"screen's matrix work ({qpad} query slots, one fp16 product per "
                             f"dimension; exact products only for blocks with a candidate) is "
                             f"{fp16_ms:.1f} ms at the dense fp16 peak; algorithmic "
                             f"fp32-equivalent rate 2 N D q (q = {nq}) {achieved:.1f} TFLOP/s",
                     "library_read": {"what": "torch.sum over the same table: one read, no "
                                              "search (context, not a ceiling)", "ms": t_read,
                                      "achieved": read_gbps, "unit": "GB/s"}},
        "sampled_check": "no row of a 200,000-row sample, other than the returned ones, "
                         "nearer than the returned k-th (exact double distances)",
        "medium_evaluation": medium,
    }
    if not args.no_cpu:
        from oracle import oracle as orc
        t0 = time.perf_counter()
        done = 0
        T = trb.S[:1_000_000].double().cpu().numpy()
        tq = 0
        while time.perf_counter() - t0 < args.cpu_budget and tq < 20:
            orc.knn(T, [tq], k)
            done += T.shape[0] - 1
            tq += 1
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": done / dt, "unit": "distances/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{tq} queries over the first 1e6 rows of the same "
                                         f"table, {dt:.1f} s single-threaded (numpy, double)"}
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="sbm100m")
    ap.add_argument("--scatter", default="sorted", choices=["sorted", "atomic"])
    ap.add_argument("--dtype", default="f32", choices=["f32", "bf16"],
                    help="element type of the tables (bf16: sorted scatter only)")
    ap.add_argument("--batches", type=int, default=64, help="distinct pre-staged batches")
    ap.add_argument("--cpu-budget", type=float, default=30.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--sequential", action="store_true",
                    help="one stream, huge_train_step per step (no overlap of grouping)")
    ap.add_argument("--no-phases", action="store_true",
                    help="diagnostic: no per-phase HIP events in the timed steps (no roofline)")
    ap.add_argument("--producer", action="store_true",
                    help="measure the random-walk sampler instead of the training step "
                         "(default workload: medium)")
    ap.add_argument("--eval", action="store_true",
                    help="time the embedding evaluation (Sec. 4: SNR, percentiles, recall) "
                         "instead of the training step")
    ap.add_argument("--knn-only", action="store_true",
                    help="with --eval: only the 100-query search over the SBM-100M table")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the step keeps both tables resident in one "
              "MI355X's HBM and has no multi-GPU path; run it with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    if args.eval:
        import torch
        torch.cuda.set_device(0)
        return bench_eval(args)

    if args.producer:
        import torch
        torch.cuda.set_device(0)
        if args.workload == "sbm100m":
            args.workload = "medium"
        return bench_producer(args)

    import numpy as np
    import torch

    import paper_2307_14490_amd as P
    from synth import make_workload

    def log(*a):
        print(*a, file=sys.stderr, flush=True)

    torch.cuda.set_device(0)
    wl = make_workload(args.workload, args.seed)
    cfg = wl.cfg
    R = max(1, args.batches)
    t0 = time.time()
    host_batches = [wl.batch(b) for b in range(R)]
    log(f"[bench] {cfg.name}: {R} batches of {cfg.batch} generated in {time.time() - t0:.1f}s")
    dev_batches = [tuple(torch.from_numpy(x).cuda() for x in b) for b in host_batches]

    tr = P.Trainer(cfg.num_nodes, cfg.dim, cfg.num_neg, cfg.batch, seed=args.seed,
                   alias_weights=wl.weights, scatter=args.scatter, dtype=args.dtype)
    torch.cuda.synchronize()
    log(f"[bench] tables initialised: 2 x {cfg.num_nodes} x {cfg.dim} {args.dtype}")
    eb = 2.0 if args.dtype == "bf16" else 4.0  # bytes per table element
    n = cfg.batch
    K = cfg.num_neg
    D = cfg.dim
    stream = torch.cuda.current_stream()

    # Per-batch distinct-row counts (sequential steps, synchronised).
    per_batch_stats = {}
    pos = 0
    if args.scatter == "sorted":
        for b in range(R):
            s, d, c = dev_batches[b]
            tr.step_no_loss(s, d, c, pos, cfg.lr)
            pos += n
            per_batch_stats[b] = tr.stats()

    # default priority, like the current stream
    side = torch.cuda.Stream()
    loss_buf = torch.zeros(1, dtype=torch.float64, device="cuda")
    # A continuous training loop: batch k+1 is prepared (on the preparation
    # stream, beside batch k's update) before batch k is applied (on the
    # current stream).  `pending` counts prepared batches not yet applied.
    state = {"pending": 0, "next_batch": 0, "pos": pos}

    def prepare_next():
        b = state["next_batch"]
        s, d, c = dev_batches[b % R]
        tr.prepare(s, d, c, state["pos"], stream=side)
        state["pos"] += n
        state["next_batch"] = b + 1
        state["pending"] += 1

    def run_steps(count, after_step=None, drain=False):
        """`count` steps, each the whole step of one batch (sampling,
        grouping, gather, loss, update, loss sum).  Pipelined, the loop keeps
        one batch prepared ahead; with drain the last step prepares none."""
        if args.sequential:
            for k in range(count):
                b = state["next_batch"]
                s, d, c = dev_batches[b % R]
                tr.step(s, d, c, state["pos"], cfg.lr, loss_out=loss_buf)
                state["pos"] += n
                state["next_batch"] = b + 1
                if after_step:
                    after_step(k)
            return
        if state["pending"] == 0:
            prepare_next()
        for k in range(count):
            if not (drain and k + 1 == count):
                prepare_next()
            tr.train_prepared(cfg.lr, loss_out=loss_buf, stream=stream)
            state["pending"] -= 1
            if after_step:
                after_step(k)

    run_steps(args.warmup)
    if tr.check() != 0:
        raise RuntimeError("device reported an error during warm-up")
    log("[bench] warm-up done")

    # Timed region: exactly K steps; the library records the fused kernel's
    # start and completion (its launch's own events, no extra queue packets)
    # on every PROFILE_EVERY-th step.
    if not args.no_phases:
        tr.profile_begin(-(-args.steps // PROFILE_EVERY), every=PROFILE_EVERY)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    side.wait_event(ev0)
    run_steps(args.steps)
    stream.wait_stream(side)  # the preparation issued for the next batch
    ev1.record(stream)
    torch.cuda.synchronize()
    total_ms = ev0.elapsed_time(ev1)
    if args.no_phases:
        log(f"[bench] no phase events: {total_ms / args.steps:.4f} ms/step")
        print(json.dumps({"metric": METRIC, "value": n * args.steps / (total_ms / 1e3),
                          "ms_per_step": total_ms / args.steps, "phases": None}), flush=True)
        return
    phase_ms, prof_steps = tr.profile_end()
    if tr.check() != 0:
        raise RuntimeError("device reported an error in the timed steps")
    ms_per_step = total_ms / args.steps
    value = n * args.steps / (total_ms / 1e3)
    log(f"[bench] {args.steps} steps in {total_ms:.2f} ms: {ms_per_step:.4f} ms/step "
        f"(last loss {loss_buf.item():.6g})")

    # Roofline probe: the rows of the same batches (sources, destinations and
    # the negatives a step would draw) read and written back unchanged, with
    # the fused kernel's launch shape and no arithmetic: the practical ceiling
    # of the step's random row traffic on this device.
    run_steps(0, drain=True)  # nothing pending: the probe may not run beside a step
    while state["pending"]:
        tr.train_prepared(cfg.lr, loss_out=loss_buf, stream=stream)
        state["pending"] -= 1
    torch.cuda.synchronize()
    pos = state["pos"]
    n_probe = min(args.steps, 50)
    for k in range(3):
        s, d, c = dev_batches[k % R]
        tr.probe_rows(s, d, pos + k * n, stream=stream)
    torch.cuda.synchronize()
    ev0.record(stream)
    for k in range(n_probe):
        s, d, c = dev_batches[k % R]
        tr.probe_rows(s, d, pos + k * n, stream=stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    probe_us = ev0.elapsed_time(ev1) / n_probe * 1e3
    if tr.check() != 0:
        raise RuntimeError("device reported an error in the probe")
    probe_bytes = 8.0 * n + 2.0 * eb * D * n * (2 + K)
    probe_gbps = probe_bytes / (probe_us * 1e-6) / 1e9
    log(f"[bench] probe: {probe_us:.1f} us per launch, {probe_gbps:.0f} GB/s")

    phases = ["setup_sample", "radix", "group", "fused_step", "finish", "loss"]
    fused_us = phase_ms[3] / max(prof_steps, 1) * 1e3
    state["pos"] = pos + 3 * n + n_probe * n
    # Phase breakdown from a separate pass of 50 steps with an event at every
    # phase boundary (those events lengthen each step by tens of microseconds,
    # so the timed steps above record only the fused kernel's two).
    n_diag = min(50, args.steps)
    tr.profile_begin(n_diag, all_phases=True)
    run_steps(n_diag, drain=True)
    stream.wait_stream(side)
    diag_ms, diag_steps = tr.profile_end()
    phase_avg_us = {p: diag_ms[i] / max(diag_steps, 1) * 1e3 for i, p in enumerate(phases)}
    del phase_avg_us["loss"]  # folded into the finish kernel

    # Distribution of step times from another separate pass: an event on the
    # apply stream after every step (a queue packet of a few microseconds
    # each); step k's time (k >= 1) is the interval between the events of
    # steps k-1 and k.
    n_dist = min(200, args.steps) + 1
    dist_ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_dist)]
    run_steps(n_dist, after_step=lambda k: dist_ev[k].record(stream), drain=True)
    stream.wait_stream(side)
    torch.cuda.synchronize()
    if tr.check() != 0:
        raise RuntimeError("device reported an error in the step-time pass")
    step_ms = np.array([dist_ev[k - 1].elapsed_time(dist_ev[k]) for k in range(1, n_dist)])
    p10, p50, p90 = (float(np.percentile(step_ms, q)) for q in (10, 50, 90))
    log(f"[bench] step time p10/p50/p90: {p10:.4f} / {p50:.4f} / {p90:.4f} ms")

    # Algorithmic bytes of the fused kernel per launch: the batch (12 B per
    # positive), each distinct row read once (eb D bytes, eb = 4 for fp32 and
    # 2 for bf16 elements) and each row that occurs once written once in
    # place.  Repeated rows are written by the duplicate kernels, not counted
    # here.
    if args.scatter == "sorted":
        seq = [(args.warmup + k) % R for k in range(args.steps)]
        seq = [b for b in seq if b in per_batch_stats]
        uS = np.mean([per_batch_stats[b][0] for b in seq])
        uT = np.mean([per_batch_stats[b][1] for b in seq])
        dup = np.mean([per_batch_stats[b][2] for b in seq])
        occ = n * (2 + K)
        kernel_bytes = 12.0 * n + eb * D * (uS + uT) + eb * D * (occ - dup)
        step_bytes = 12.0 * n + 2.0 * eb * D * (uS + uT)
    else:
        uS = uT = dup = None
        kernel_bytes = 12.0 * n + 4.0 * D * n * (2 + K)  # gather kernel: every row read
        step_bytes = 12.0 * n + 8.0 * D * n * (2 + K)
    achieved = kernel_bytes / (fused_us * 1e-6) / 1e9
    traffic = read_traffic(cfg.name, args.dtype) if args.scatter == "sorted" else None
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "positives/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",  # the arithmetic type (bf16 tables compute in fp32)
        "data": "synthetic",
        "config": {
            "workload": cfg.name,
            "num_nodes": cfg.num_nodes,
            "dim": D,
            "num_neg_per_pos": K,
            "batch": n,
            "negatives": cfg.neg_kind,
            "scatter": args.scatter,
            "tables": args.dtype,
            "lr": cfg.lr,
            "staged_batches": R,
            "grouping": ("sequential" if args.sequential else
                         "on a preparation stream, beside the previous batch's update"),
        },
        "roofline": {
            "kernel": KERNEL if args.scatter == "sorted" else "k_atomic_gather",
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "avg_kernel_us": fused_us,
            "timed_launches": prof_steps,
            "timing": f"HIP events at the fused kernel's start and completion (its launch's "
                      f"own events) on every {PROFILE_EVERY}th timed step",
            "alg_bytes_per_launch": kernel_bytes,
            "probe": {
                "achieved": probe_gbps,
                "unit": "GB/s",
                "avg_us": probe_us,
                "bytes_per_launch": probe_bytes,
                "what": "the same batches' rows read and written back unchanged, no arithmetic",
            },
            "frac_of_probe": achieved / probe_gbps,
        },
        "step": {
            "alg_bytes": step_bytes,
            "alg_GBps": step_bytes / (ms_per_step * 1e-3) / 1e9,
            "phase_avg_us": phase_avg_us,
            "phase_note": "from a separate 50-step pass with an event at every phase boundary",
            "ms_percentiles": {"p10": p10, "p50": p50, "p90": p90, "steps": int(step_ms.size),
                               "positives_per_s_at_p50": n / (p50 * 1e-3),
                               "note": "a separate pass with one event after every step"},
            "unique_src_rows": uS,
            "unique_ctx_rows": uT,
            "repeated_row_occurrences": dup,
        },
    }
    tr.close()
    del tr, dev_batches
    torch.cuda.empty_cache()
    if not args.no_cpu:
        log("[bench] timing the CPU oracle on a sample")
        out["cpu_baseline"] = cpu_baseline(wl, args.seed, budget_s=args.cpu_budget)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
