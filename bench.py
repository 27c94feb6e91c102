"""Benchmark: threshold-aware IVF search (W = 8, lookahead) on one MI355X.

One step = one sieve_search call over the workload's whole query batch with
inputs resident in HBM: centroid ranking, partition-major scheduling rounds,
the partition scan with the tau test, the stop-rule updates and the final
top-k.  The default workload is the mid-size self-join (N = 1,000,000 rows,
d = 128, fp32, nlist = 1,024, Q = 10,000, k = 10, tau = 0.92, W = 8,
nprobe_max = 128).  The same run times the fixed-probe baseline (nprobe = 128)
on the same GPU for the speedup, reads the partition-scan kernel's device
time from the library's HIP events on the search stream for the roofline,
and times the CPU oracle on a bounded query sample (cpu_baseline).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config c2]

Prints exactly one JSON line (last line of stdout).
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

HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"f32": 157.3, "f16": 2500.0}
PMC_FILE = os.path.join(ROOT, "profiles", "scan_traffic_pmc.json")
# oracle sample per workload: roughly 10-30 s of single-thread fp64 work
ORACLE_SAMPLE = {"tiny": 150, "tiny16": 150, "c1": 1000, "c2": 10000, "c3": 200, "c5": 300}
SCAN_SOURCES = ["paper_2608_03199_amd/csrc/scan.hip", "paper_2608_03199_amd/csrc/mfma_tile.h"]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def scan_source_hash() -> str:
    h = hashlib.sha256()
    for p in SCAN_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(config: str):
    """HBM bytes per scan launch from the committed rocprofv3 counter summary,
    or None when it is absent or was taken on a different scan kernel."""
    try:
        with open(PMC_FILE) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    e = d.get(config)
    if not e or e.get("scan_source_hash") != scan_source_hash():
        return None
    return e.get("bytes_per_launch")


def workload_name(spec) -> str:
    return (f"{spec.name}: self-join N={spec.n:,} d={spec.d} {spec.dtype}, nlist={spec.nlist:,}, "
            f"Q={spec.nq:,}, k={spec.k}, tau={spec.tau}, W={spec.W}, "
            f"nprobe_max={spec.nprobe_max}, lookahead on")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c2")
    ap.add_argument("--oracle-queries", type=int, default=None,
                    help="queries in the single-thread oracle sample (default: about 10-30 s "
                         "of oracle work for the workload)")
    ap.add_argument("--no-oracle", action="store_true")
    ap.add_argument("--skip-fixed", action="store_true",
                    help="do not time the fixed-probe baseline (profiling runs)")
    ap.add_argument("--skip-calibrated", action="store_true",
                    help="do not time the in-call calibrated search (profiling runs)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 1 GiB device copy (HBM counter calibration)")
    ap.add_argument("--envelope", action="store_true",
                    help="k in {5, 10, 20, 50} and tau in {0.10 .. 0.90} on the 1M x 128 data: "
                         "queries/s, speedup over fixed probing, candidates, overlap with the "
                         "fixed-probe output (one JSON line)")
    ap.add_argument("--concurrency", action="store_true",
                    help="queries per call in {1, 10, 100, 1000, 10000} on the 1M x 128 data, "
                         "for lookahead, basic and serial dispatch and fixed probing (one JSON "
                         "line)")
    ap.add_argument("--multi", action="store_true",
                    help="multi-index search: the 100M x 128 data split into 16 coarse shards, "
                         "each its own IVF with its own stop rule, one global top-k; against "
                         "fixed probing of every shard (one JSON line)")
    ap.add_argument("--multi-shards", type=int, default=16)
    ap.add_argument("--multi-nprobe", type=int, default=64,
                    help="per-shard nprobe of the fixed baseline and per-shard cap of the "
                         "threshold search")
    ap.add_argument("--sweep", action="store_true",
                    help="W / lookahead / tau / fixed-nprobe sweep with recall on the 1M x 128 "
                         "data (prints one JSON line with the table)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: this build measures one GPU only; --gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2608_03199_amd as ps
    import sieve_workloads as sw

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.sweep:
        return sweep(args, ps, sw, np, torch, dev)
    if args.envelope:
        return envelope(args, ps, sw, np, torch, dev)
    if args.concurrency:
        return concurrency(args, ps, sw, np, torch, dev)
    if args.multi:
        return multi(args, ps, sw, np, torch, dev)
    spec = sw.SPECS[args.config]
    log(f"[bench] generating {args.config} on {dev}")
    t0 = time.time()
    w = sw.make(spec, device=dev)
    torch.cuda.synchronize()
    log(f"[bench] generated in {time.time() - t0:.1f}s; lists {sw.list_stats(w.list_offsets.cpu().numpy())}")
    ix = ps.Index(w.vectors, w.list_offsets, w.ids, w.centroids)
    nq = spec.nq

    if args.copy_probe:
        # 1 GiB fill (writes 1 GiB) and 1 GiB elementwise scale (reads 1 GiB,
        # writes 1 GiB): the HBM byte counters of these two kernels calibrate
        # the counters read on the scan kernel.
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        a.fill_(1.0)
        torch.mul(a, 2.0, out=b)
        torch.cuda.synchronize()
        del a, b

    def sieve(with_stats=True):
        return ix.search(w.queries, w.exclude_ids, spec.k, spec.tau, spec.W, spec.nprobe_max,
                         lookahead=True, with_stats=with_stats)

    def fixed(with_stats=True):
        return ix.search_fixed(w.queries, w.exclude_ids, spec.k, spec.tau, spec.fixed_nprobe,
                               with_stats=with_stats)

    for _ in range(args.warmup):
        sieve()
        if not args.skip_fixed:
            fixed()
    torch.cuda.synchronize()

    # timed region: exactly K sieve steps
    log(f"[bench] timing {args.steps} steps")
    stats = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        r = sieve()
        stats.append(r[3])
    torch.cuda.synchronize()
    t_sieve = time.perf_counter() - t0
    ids, scores, probes = r[0], r[1], r[2]

    # fixed-probe baseline on the same GPU (same number of steps)
    fstats = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(0 if args.skip_fixed else args.steps):
        fr = fixed()
        fstats.append(fr[3])
    torch.cuda.synchronize()
    t_fixed = time.perf_counter() - t0 if not args.skip_fixed else float("nan")

    # in-call calibration (Appendix A): a seeded 2% sample fully probed, the
    # window chosen for a 0.5% sample-relative loss target, the rest searched
    # with it; the sample's full probing is inside the timed region
    cal = None
    if not args.skip_calibrated:
        ns = max(1, nq // 50)
        smp = torch.from_numpy(np.random.default_rng(spec.seed + 91).choice(
            nq, ns, replace=False).astype(np.int32)).to(dev)

        def calibrated(with_stats=True):
            return ix.search_calibrated(w.queries, w.exclude_ids, spec.k, spec.tau,
                                        spec.nprobe_max, smp, CAL_EPS, spec.W,
                                        with_stats=with_stats)

        calibrated()
        csteps = max(1, min(args.steps, 5))
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(csteps):
            cr = calibrated()
        torch.cuda.synchronize()
        t_cal = (time.perf_counter() - t0) / csteps
        cal = {"W": cr[3], "sample": ns, "eps": CAL_EPS, "steps": csteps,
               "qps": round(nq / t_cal, 1),
               "speedup_vs_fixed": (None if args.skip_fixed else
                                    round((t_fixed / args.steps) / t_cal, 3)),
               "mean_probes": round(float(cr[2].float().mean().item()), 3)}

    ms_step = 1e3 * t_sieve / args.steps
    qps = nq * args.steps / t_sieve
    fixed_qps = nq * args.steps / t_fixed
    st = stats[-1]
    mean = lambda xs, f: float(np.mean([getattr(x, f) for x in xs]))
    ms_scan = mean(stats, "ms_scan")
    launches = st.scan_launches
    bytes_launch = st.scan_bytes / max(launches, 1)
    flops_launch = st.scan_flops / max(launches, 1)
    avg_launch_ms = ms_scan / max(launches, 1)
    peak_f = MFMA_PEAK_TFLOPS[spec.dtype]
    t_hbm = st.scan_bytes / (HBM_PEAK_GBS * 1e9)
    t_mfma = st.scan_flops / (peak_f * 1e12)
    bound = "hbm" if t_hbm >= t_mfma else "mfma"
    gbs = bytes_launch / (avg_launch_ms * 1e-3) / 1e9
    tfs = flops_launch / (avg_launch_ms * 1e-3) / 1e12
    traffic = measured_traffic(args.config)
    if bound == "hbm":
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4)}
    else:
        roof = {"bound": "mfma", "achieved": round(tfs, 2), "peak": peak_f, "unit": "TFLOP/s",
                "frac": round(tfs / peak_f, 4)}
    roof["traffic"] = traffic
    roof["kernel"] = "scan_kernel (partition scan + tau test)"
    roof["launches_per_step"] = launches
    roof["avg_launch_ms"] = round(avg_launch_ms, 5)
    roof["alg_bytes_per_launch"] = round(bytes_launch)
    roof["alg_flops_per_launch"] = round(flops_launch)
    roof["other_bound_frac"] = round((tfs / peak_f) if bound == "hbm" else (gbs / HBM_PEAK_GBS), 4)
    roof["roofline_time_frac"] = round(max(t_hbm, t_mfma) / (ms_scan * 1e-3), 4)

    out = {
        "metric": "queries/sec at W=8 (k=10, tau); speedup vs fixed-nprobe; scan HBM GB/s",
        "value": round(qps, 1),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic (seeded mixture + near-duplicate groups, spherical k-means IVF)",
        "config": {"workload": workload_name(spec), "queries": nq, "k": spec.k,
                   "tau": spec.tau, "W": spec.W, "nprobe_max": spec.nprobe_max,
                   "fixed_nprobe": spec.fixed_nprobe, "parallelism": "single GPU"},
        "speedup_vs_fixed": None if args.skip_fixed else round(t_fixed / t_sieve, 3),
        "fixed_qps": None if args.skip_fixed else round(fixed_qps, 1),
        "partition_vectors_per_s": round(st.vectors_scanned * args.steps / t_sieve, 1),
        "scan_hbm_gbs": round(gbs, 1),
        "mean_probes": round(float(probes.float().mean().item()), 3),
        "scanned_probes_per_query": round(st.items / nq, 3),
        "rounds": st.rounds,
        "phase_ms": {k: round(mean(stats, "ms_" + k), 4) for k in
                     ("rank", "sched", "scan", "update", "finalize", "total")},
        "fixed_phase_ms": ({k: round(mean(fstats, "ms_" + k), 4) for k in
                            ("rank", "sched", "scan", "finalize", "total")} if fstats else None),
        "roofline": roof,
        "calibrated": cal,
    }

    if not args.no_oracle:
        import oracle
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from parity import compare
        h = w.numpy()
        m = min(args.oracle_queries or ORACLE_SAMPLE.get(args.config, 1000), nq)
        rng = np.random.default_rng(spec.seed + 77)
        sel = np.sort(rng.choice(nq, m, replace=False))
        log(f"[bench] oracle on {m} queries, 1 thread")
        t0 = time.perf_counter()
        o = oracle.search(h["vectors"], h["list_offsets"], h["ids"], h["centroids"],
                          h["queries"][sel], h["exclude_ids"][sel], spec.k, spec.tau, spec.W,
                          spec.nprobe_max, oracle.MODE_A, 1)
        t_or = time.perf_counter() - t0
        rep = compare(ids.cpu().numpy()[sel], scores.cpu().numpy()[sel],
                      probes.cpu().numpy()[sel], o)
        out["cpu_baseline"] = {"value": round(m / t_or, 2), "unit": "queries/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{m} seeded queries of the same workload, "
                                         f"single thread, {t_or:.1f}s",
                               "cpu": _cpu_model()}
        out["parity_sample"] = {k: rep[k] for k in ("queries", "mismatch", "flag_tau_edge",
                                                    "flag_kth_tie", "flagged_mismatch",
                                                    "max_score_err")}
    ix.close()
    print(json.dumps(out), flush=True)


W_INF = 0x7FFFFFFF
CAL_EPS = 0.005  # sample-relative loss target of the calibrated leg (Appendix A)


def sweep(args, ps, sw, np, torch, dev):
    """Operating sweep on the 1M x 128 fp32 data: W in {2, 4, 8, 16, inf} with lookahead on
    and off (outputs must be identical), fixed nprobe in {32, 64, 128, 256}, each at tau in
    {0.90, 0.95, 0.98}; queries/s over the whole 10,000-query batch, mean probes, and pooled
    filtered top-10 recall (Sec. 6.1) on a seeded 2,000-query subset against exact filtered
    brute force from the oracle (W = inf, nprobe = nlist)."""
    import oracle
    from sieve_workloads.metrics import pooled_recall
    spec = sw.SPECS["c2"]
    log("[sweep] generating c2")
    w = sw.make(spec, device=dev)
    ix = ps.Index(w.vectors, w.list_offsets, w.ids, w.centroids)
    rng = np.random.default_rng(spec.seed + 4)
    sel = np.sort(rng.choice(spec.nq, 2000, replace=False))
    h = w.numpy()
    steps = max(1, args.steps // 4)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            r = fn()
        torch.cuda.synchronize()
        return r, (time.perf_counter() - t0) / steps

    # exact filtered top-10 at the lowest tau; a higher tau keeps the prefix whose fp64
    # score reaches it (the top-10 order does not depend on tau)
    log("[sweep] exact filtered top-10 of 2,000 queries (oracle brute force)")
    exact = oracle.bruteforce(h["vectors"], h["ids"], h["queries"][sel], h["exclude_ids"][sel],
                              spec.k, 0.90, os.cpu_count() or 1)
    rows = []
    for tau in (0.90, 0.95, 0.98):
        truth_ids = np.where(exact.scores >= tau, exact.ids, -1)
        for W in (2, 4, 8, 16, W_INF):
            res = {}
            for la in (True, False):
                r, sec = timed(lambda: ix.search(w.queries, w.exclude_ids, spec.k, tau, W,
                                                 spec.nprobe_max, lookahead=la))
                res[la] = (r, sec)
            a, b = res[True][0], res[False][0]
            same = all(bool(torch.equal(x, y)) for x, y in zip(a, b))
            ids = a[0].cpu().numpy()
            rec = pooled_recall(ids[sel], truth_ids)[0]
            rows.append({"mode": "sieve", "tau": tau, "W": "inf" if W == W_INF else W,
                         "qps_lookahead": round(spec.nq / res[True][1], 1),
                         "qps_no_lookahead": round(spec.nq / res[False][1], 1),
                         "lookahead_identical": same,
                         "mean_probes": round(float(a[2].float().mean()), 3),
                         "recall_at_10": round(rec, 5)})
            log(f"[sweep] {rows[-1]}")
        for npb in (32, 64, 128, 256):
            r, sec = timed(lambda: ix.search_fixed(w.queries, w.exclude_ids, spec.k, tau, npb))
            ids = r[0].cpu().numpy()
            rows.append({"mode": "fixed", "tau": tau, "nprobe": npb,
                         "qps": round(spec.nq / sec, 1), "mean_probes": float(npb),
                         "recall_at_10": round(pooled_recall(ids[sel], truth_ids)[0], 5)})
            log(f"[sweep] {rows[-1]}")
    ix.close()
    out = {"metric": "operating sweep: queries/s, mean probes, pooled filtered recall@10",
           "config": {"workload": workload_name(spec), "recall_subset": 2000,
                      "nprobe_max": spec.nprobe_max},
           "steps_per_point": steps, "sweep": rows}
    print(json.dumps(out), flush=True)


def _timed(torch, fn, steps):
    fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        r = fn()
    torch.cuda.synchronize()
    return r, (time.perf_counter() - t0) / steps


def envelope(args, ps, sw, np, torch, dev):
    """Operating envelope on the 1M x 128 fp32 data (Sec. 6.4: thresholds down to 0.10, k up
    to 50): W = 8 with lookahead against fixed nprobe = 128 on the whole 10,000-query batch;
    overlap = pooled fraction of the fixed-probe result that the threshold search returns."""
    spec = sw.SPECS["c2"]
    log("[envelope] generating c2")
    w = sw.make(spec, device=dev)
    ix = ps.Index(w.vectors, w.list_offsets, w.ids, w.centroids)
    steps = max(1, args.steps // 4)
    rows = []
    points = [(k, spec.tau) for k in (5, 10, 20, 50)] + \
             [(spec.k, t) for t in (0.10, 0.30, 0.50, 0.70, 0.90)]
    for k, tau in points:
        r, sec = _timed(torch, lambda: ix.search(w.queries, w.exclude_ids, k, tau, spec.W,
                                                 spec.nprobe_max, with_stats=True), steps)
        f, fsec = _timed(torch, lambda: ix.search_fixed(w.queries, w.exclude_ids, k, tau,
                                                        spec.fixed_nprobe), steps)
        a, b = r[0].cpu().numpy(), f[0].cpu().numpy()
        tot = int((b >= 0).sum())
        kept = sum(len(set(x[x >= 0].tolist()) & set(y[y >= 0].tolist())) for x, y in zip(a, b))
        rows.append({"k": k, "tau": tau, "qps": round(spec.nq / sec, 1),
                     "fixed_qps": round(spec.nq / fsec, 1), "speedup": round(fsec / sec, 3),
                     "mean_probes": round(float(r[2].float().mean()), 3),
                     "scanned_probes_per_query": round(r[3].items / spec.nq, 3),
                     "candidates": int(r[3].hits), "rounds": int(r[3].rounds),
                     "overlap_with_fixed": round(kept / tot, 5) if tot else None})
        log(f"[envelope] {rows[-1]}")
    ix.close()
    out = {"metric": "operating envelope: queries/s and speedup over fixed probing",
           "config": {"workload": workload_name(spec), "W": spec.W,
                      "fixed_nprobe": spec.fixed_nprobe},
           "steps_per_point": steps, "envelope": rows}
    print(json.dumps(out), flush=True)


def concurrency(args, ps, sw, np, torch, dev):
    """Queries per call (Sec. 6.4's request-size sweep) on the 1M x 128 fp32 data, W = 8:
    lookahead, basic (Algorithm 1) and serial dispatch.  Each point issues consecutive calls
    over a prefix of the 10,000-query batch (at most 200 calls) and reports queries/s."""
    spec = sw.SPECS["c2"]
    log("[concurrency] generating c2")
    w = sw.make(spec, device=dev)
    ix = ps.Index(w.vectors, w.list_offsets, w.ids, w.centroids)
    rows = []
    for per in (1, 10, 100, 1000, 10000):
        calls = min(200, spec.nq // per)
        row = {"queries_per_call": per, "calls": calls}
        for name, kw in (("lookahead", dict(lookahead=True)), ("basic", dict(lookahead=False)),
                         ("serial", dict(serial=True)), ("fixed", None)):
            def run():
                for c in range(calls):
                    q0 = c * per
                    q, ex = w.queries[q0:q0 + per], w.exclude_ids[q0:q0 + per]
                    if kw is None:
                        r = ix.search_fixed(q, ex, spec.k, spec.tau, spec.fixed_nprobe)
                    else:
                        r = ix.search(q, ex, spec.k, spec.tau, spec.W, spec.nprobe_max, **kw)
                return r
            _, sec = _timed(torch, run, 1)
            row[name + "_qps"] = round(calls * per / sec, 1)
        row["lookahead_vs_fixed"] = round(row["lookahead_qps"] / row["fixed_qps"], 3)
        row["basic_vs_fixed"] = round(row["basic_qps"] / row["fixed_qps"], 3)
        row["serial_vs_fixed"] = round(row["serial_qps"] / row["fixed_qps"], 3)
        rows.append(row)
        log(f"[concurrency] {row}")
    ix.close()
    out = {"metric": "queries/s by queries per call (W=8): lookahead, basic and serial dispatch, "
                     "and fixed probing",
           "config": {"workload": workload_name(spec), "W": spec.W,
                      "nprobe_max": spec.nprobe_max},
           "concurrency": rows}
    print(json.dumps(out), flush=True)


def _coarse_groups(torch, centroids, groups, iters=15, seed=7):
    """Lloyd's k-means over the list centroids (fp32, seeded): each list goes to one coarse
    group, so each group is a set of whole lists."""
    c = centroids.float()
    g = torch.Generator(device=c.device).manual_seed(seed)
    cen = c[torch.randperm(c.shape[0], generator=g, device=c.device)[:groups]].clone()
    for _ in range(iters):
        a = torch.argmax(c @ cen.T, dim=1)
        for j in range(groups):
            m = a == j
            if bool(m.any()):
                v = c[m].sum(0)
                cen[j] = v / v.norm().clamp_min(1e-12)
    return torch.argmax(c @ cen.T, dim=1)


def multi(args, ps, sw, np, torch, dev):
    """Multi-index search (Sec. 6.1's public 100M layout: coarse k-means shards, each with its
    own IVF; every shard searched with its own stop rule, one global top-k merge) on one GPU.
    The 100M x 128 fp16 data's lists are grouped into coarse shards by k-means over their
    centroids; each shard keeps its lists (so every row stays with its nearest centroid).
    Threshold search W = 8 with lookahead, per-shard cap = the fixed baseline's per-shard
    nprobe; overlap = pooled fraction of the fixed-probe output returned."""
    spec = sw.SPECS["c5"]
    S, P = args.multi_shards, args.multi_nprobe
    log(f"[multi] generating c5 on {dev}")
    w = sw.make(spec, device=dev)
    off = w.list_offsets
    counts = off[1:] - off[:-1]
    grp = _coarse_groups(torch, w.centroids, S)
    row_grp = torch.repeat_interleave(grp, counts)
    ixs, sizes = [], []
    for j in range(S):
        lists = torch.nonzero(grp == j).flatten()
        if lists.numel() == 0:
            continue
        rows = torch.nonzero(row_grp == j).flatten()  # ascending: lists stay whole, in order
        loff = torch.zeros(lists.numel() + 1, dtype=torch.int64, device=dev)
        loff[1:] = torch.cumsum(counts[lists], 0)
        ixs.append(ps.Index(w.vectors[rows], loff, w.ids[rows], w.centroids[lists]))
        sizes.append((int(lists.numel()), int(rows.numel())))
        del rows, loff
    del row_grp
    torch.cuda.synchronize()
    log(f"[multi] {len(ixs)} shards (lists, rows): {sizes}")
    steps = max(1, args.steps // 4)
    r, sec = _timed(torch, lambda: ps.search_multi(ixs, w.queries, w.exclude_ids, spec.k,
                                                   spec.tau, spec.W, P, with_stats=True), steps)
    f, fsec = _timed(torch, lambda: ps.search_multi(ixs, w.queries, w.exclude_ids, spec.k,
                                                    spec.tau, 0x7FFFFFFF, P), steps)
    a, b = r[0].cpu().numpy(), f[0].cpu().numpy()
    tot = int((b >= 0).sum())
    kept = int(sum(np.intersect1d(x[x >= 0], y[y >= 0]).size for x, y in zip(a, b)))
    st = r[3]
    row = {"shards": len(ixs), "per_shard_nprobe": P, "qps": round(spec.nq / sec, 1),
           "fixed_qps": round(spec.nq / fsec, 1), "speedup": round(fsec / sec, 3),
           "mean_probes": round(float(r[2].double().mean()), 3),
           "fixed_probes": int(f[2][0]), "candidates": int(st.hits),
           "overlap_with_fixed": round(kept / tot, 5) if tot else None,
           "ms_rank": round(st.ms_rank, 2), "ms_scan": round(st.ms_scan, 2),
           "ms_total": round(st.ms_total, 2)}
    log(f"[multi] {row}")
    for ix in ixs:
        ix.close()
    out = {"metric": "multi-index threshold search: queries/s and speedup over fixed probing",
           "config": {"workload": workload_name(spec), "shards": len(ixs),
                      "shard_lists": [x[0] for x in sizes], "shard_rows": [x[1] for x in sizes],
                      "W": spec.W, "per_shard_nprobe": P},
           "steps": steps, "multi": row}
    print(json.dumps(out), flush=True)


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip() + f" ({os.cpu_count()} threads visible)"
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    main()
