"""Benchmark: threshold-aware IVF search (W = 8) on one MI355X, every workload in one run.

One step = one sieve_search call over a workload's whole query batch with inputs resident in
HBM: centroid ranking, partition-major scheduling rounds, the partition scan with the tau test,
the stop-rule updates and the final top-k.  The headline (`value`, `config`, `roofline`,
`cpu_baseline`) is the largest workload, the 100M x 128 fp16 self-join (nlist 16,384, 1M
queries, k = 10, tau = 0.90, W = 8, nprobe_max = 512), searched with Algorithm 2 lookahead
(committed ranks only); the smaller workloads are reported under `configs` from the same run.
Per workload the run also times:
  * speculative issue (the library's addition to Algorithm 2; identical outputs),
  * the fixed-probe baseline at the workload's nprobe on the same GPU (speedup),
  * the in-call calibrated search (Appendix A),
  * the CPU oracle: one thread on a small seeded sample, and all host threads (at most 16)
    on the seeded parity subset, whose GPU results are compared with it element by element.
The partition scan's device time per round comes from the library's HIP events on the search
stream (sieve_round_log), over the timed steps.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config all|c1|c2|c3|c5]

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
CONFIG_ORDER = ["c1", "c2", "c3", "c5"]
# single-thread oracle sample per workload: roughly 5-15 s of fp64 work
ORACLE_ONE_THREAD = {"tiny": 150, "tiny16": 150, "c1": 1000, "c2": 4000, "c3": 100, "c5": 150}
# parity subset, checked with the threaded oracle (all queries of the small workloads)
ORACLE_PARITY = {"tiny": 150, "tiny16": 150, "c1": 1000, "c2": 10000, "c3": 5000, "c5": 5000}
ORACLE_MAX_THREADS = 16
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
            f"nprobe_max={spec.nprobe_max}, Algorithm 2 lookahead")


def roofline(dtype, rounds, config):
    """Roofline of the partition scan over the timed steps' rounds.

    Step-aggregate form (`frac`): the summed algorithmic bytes and flops of a step priced
    against the bound they imply, achieved = per-launch work / average launch time.
    Per-round form (`frac_rounds`): sum over rounds of max(B_r / BW, F_r / P) divided by
    the summed measured scan time, each round against its own bound."""
    peak_f = MFMA_PEAK_TFLOPS[dtype]
    launches = len(rounds)
    B = sum(r["scan_bytes"] for r in rounds)
    F = sum(r["scan_flops"] for r in rounds)
    T = sum(r["ms_scan"] for r in rounds) * 1e-3
    t_hbm = B / (HBM_PEAK_GBS * 1e9)
    t_mfma = F / (peak_f * 1e12)
    bound = "hbm" if t_hbm >= t_mfma else "mfma"
    avg_s = T / max(launches, 1)
    gbs = (B / max(launches, 1)) / avg_s / 1e9 if avg_s > 0 else 0.0
    tfs = (F / max(launches, 1)) / avg_s / 1e12 if avg_s > 0 else 0.0
    if bound == "hbm":
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4)}
    else:
        roof = {"bound": "mfma", "achieved": round(tfs, 2), "peak": peak_f, "unit": "TFLOP/s",
                "frac": round(tfs / peak_f, 4)}
    roof["traffic"] = measured_traffic(config)
    roof["kernel"] = "scan_kernel (partition scan + tau test)"
    roof["launches_per_step"] = launches
    roof["avg_launch_ms"] = round(avg_s * 1e3, 5)
    roof["alg_bytes_per_launch"] = round(B / max(launches, 1))
    roof["alg_flops_per_launch"] = round(F / max(launches, 1))
    roof["other_bound_frac"] = round((tfs / peak_f) if bound == "hbm" else (gbs / HBM_PEAK_GBS),
                                     4)
    per, tstar_sum = [], 0.0
    for r in rounds:
        tb = r["scan_bytes"] / (HBM_PEAK_GBS * 1e9)
        tf = r["scan_flops"] / (peak_f * 1e12)
        ts = max(tb, tf)
        tstar_sum += ts
        t = r["ms_scan"] * 1e-3
        per.append({"items": r["items"], "list_loads": r["list_loads"],
                    "bytes": round(r["scan_bytes"]), "flops": round(r["scan_flops"]),
                    "ms": round(r["ms_scan"], 4), "bound": "hbm" if tb >= tf else "mfma",
                    "bound_ms": round(ts * 1e3, 4), "frac": round(ts / t, 4) if t > 0 else None})
    roof["frac_rounds"] = round(tstar_sum / T, 4) if T > 0 else None
    roof["rounds"] = per
    return roof


def e1_diagnostics(np, ids, probes, W, n):
    """The paper's Figure 1 analogue from the outputs: the share of queries without a
    neighbour, and the last-hit rank L of the others (probes = min(L + W, n), so L is
    probes - W wherever the query stopped before n)."""
    zero = float((ids[:, 0] < 0).mean())
    p = probes.astype(np.int64)
    stopped = p < n
    L = np.where(stopped, p - W, -1)
    with_hit = L[(L > 0)]
    pct = {f"p{q}": (int(np.percentile(with_hit, q)) if with_hit.size else None)
           for q in (50, 90, 99)}
    return {"zero_neighbour_share": round(zero, 5),
            "last_hit_rank": dict(pct, max=int(with_hit.max()) if with_hit.size else None,
                                  queries=int(with_hit.size)),
            "reached_nprobe_max": int((~stopped).sum())}


def _timed_steps(torch, fn, steps):
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    out = []
    for _ in range(steps):
        out.append(fn())
    torch.cuda.synchronize()
    return out, time.perf_counter() - t0


def run_config(name, args, ps, sw, np, torch, dev, headline):
    spec = sw.SPECS[name]
    log(f"[bench] {name}: generating on {dev}")
    t0 = time.time()
    w = sw.make(spec, device=dev)
    torch.cuda.synchronize()
    lists = sw.list_stats(w.list_offsets.cpu().numpy())
    log(f"[bench] {name}: generated in {time.time() - t0:.1f}s; lists {lists}")
    ix = ps.Index(w.vectors, w.list_offsets, w.ids, w.centroids)
    nq = spec.nq
    K = args.steps

    def sieve(with_stats=True, speculative=False):
        return ix.search(w.queries, w.exclude_ids, spec.k, spec.tau, spec.W, spec.nprobe_max,
                         lookahead=True, speculative=speculative, with_stats=with_stats)

    def fixed(with_stats=True):
        return ix.search_fixed(w.queries, w.exclude_ids, spec.k, spec.tau, spec.fixed_nprobe,
                               with_stats=with_stats)

    if args.copy_probe:
        # 1 GiB fill (writes 1 GiB) and 1 GiB elementwise scale (reads 1 GiB, writes 1 GiB):
        # the HBM byte counters of these two kernels calibrate the scan kernel's counters.
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        a.fill_(1.0)
        torch.mul(a, 2.0, out=b)
        torch.cuda.synchronize()
        del a, b

    for _ in range(args.warmup):
        sieve()
    # timed region: exactly K steps of the threshold search (Algorithm 2 lookahead); the
    # per-round scan times of every step come from the library's event log
    log(f"[bench] {name}: timing {K} steps")
    rounds = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        r = sieve()
        rounds.extend(x.as_dict() for x in ix.round_log())
    torch.cuda.synchronize()
    t_sieve = time.perf_counter() - t0
    ids, scores, probes, st = r
    stats = st
    res = {"workload": workload_name(spec), "queries": nq, "steps": K,
           "qps": round(nq * K / t_sieve, 1), "ms_per_step": round(1e3 * t_sieve / K, 4),
           "mean_probes": round(float(probes.float().mean().item()), 3),
           "scanned_probes_per_query": round(stats.items / nq, 3), "rounds": stats.rounds,
           "partition_vectors_per_s": round(stats.vectors_scanned * K / t_sieve, 1),
           "candidates": int(stats.hits), "pool_entries": int(stats.pool_entries),
           "heavy_records": int(stats.heavy_records)}
    roof = roofline(spec.dtype, rounds, name)
    # per-step round table: the last step's rounds (every step runs the same rounds)
    roof["rounds"] = roof["rounds"][-stats.rounds:] if stats.rounds else []
    res["scan_hbm_gbs"] = round(sum(x["scan_bytes"] for x in rounds) /
                                max(sum(x["ms_scan"] for x in rounds) * 1e-3, 1e-12) / 1e9, 1)
    res["phase_ms"] = {k: round(getattr(stats, "ms_" + k), 4) for k in
                       ("rank", "sched", "scan", "update", "finalize", "total")}
    res["roofline"] = roof
    res["lists"] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in lists.items()}
    h_ids, h_probes = ids.cpu().numpy(), probes.cpu().numpy()
    res["e1"] = e1_diagnostics(np, h_ids, h_probes, spec.W, min(spec.nprobe_max, spec.nlist))

    if args.sieve_only:
        # counter runs: the threshold-search steps alone (no other scan launches follow)
        ix.close()
        del w
        torch.cuda.empty_cache()
        return res

    # speculative issue past the stop line (same outputs, fewer rounds, more searches)
    ks = max(1, min(K, 5))
    sp, t_sp = _timed_steps(torch, lambda: sieve(speculative=True), ks)
    same = all(bool(torch.equal(x, y)) for x, y in zip(sp[-1][:3], (ids, scores, probes)))
    res["speculative"] = {"qps": round(nq * ks / t_sp, 1), "steps": ks,
                          "rounds": sp[-1][3].rounds,
                          "scanned_probes_per_query": round(sp[-1][3].items / nq, 3),
                          "identical_outputs": same}

    # fixed-probe baseline on the same GPU
    kf = K if spec.n <= 1_000_000 else max(1, min(K, 3))
    fixed()
    fr, t_fixed = _timed_steps(torch, fixed, kf)
    fst = fr[-1][3]
    res["fixed_nprobe"] = spec.fixed_nprobe
    res["fixed_qps"] = round(nq * kf / t_fixed, 1)
    res["speedup_vs_fixed"] = round((t_fixed / kf) / (t_sieve / K), 3)
    res["speculative"]["speedup_vs_fixed"] = round((t_fixed / kf) / (t_sp / ks), 3)
    res["fixed_phase_ms"] = {k: round(getattr(fst, "ms_" + k), 4) for k in
                             ("rank", "sched", "scan", "finalize", "total")}
    res["fixed_roofline"] = {k: v for k, v in roofline(
        spec.dtype, [x.as_dict() for x in ix.round_log()], name).items()
        if k not in ("rounds", "traffic")}

    # in-call calibration (Appendix A): a seeded 2% sample fully probed, the window chosen
    # for a 0.5% sample-relative loss target, the rest searched with it; the sample's full
    # probing is inside the timed region
    if not args.skip_calibrated:
        ns = max(1, nq // 50)
        smp = torch.from_numpy(np.random.default_rng(spec.seed + 91).choice(
            nq, ns, replace=False).astype(np.int32)).to(dev)
        cal_fn = lambda: ix.search_calibrated(w.queries, w.exclude_ids, spec.k, spec.tau,
                                              spec.nprobe_max, smp, CAL_EPS, spec.W)
        cal_fn()
        kc = max(1, min(K, 3))
        cr, t_cal = _timed_steps(torch, cal_fn, kc)
        res["calibrated"] = {"W": cr[-1][3], "sample": ns, "eps": CAL_EPS, "steps": kc,
                             "qps": round(nq * kc / t_cal, 1),
                             "speedup_vs_fixed": round((t_fixed / kf) / (t_cal / kc), 3),
                             "mean_probes": round(float(cr[-1][2].float().mean().item()), 3)}
    ix.close()

    if not args.no_oracle:
        res.update(oracle_legs(name, spec, w, np, h_ids, scores.cpu().numpy(), h_probes, args))
    del w, ids, scores, probes
    torch.cuda.empty_cache()
    return res


def oracle_legs(name, spec, w, np, ids, scores, probes, args):
    """cpu_baseline: the oracle (mode A) on one thread over a small seeded sample, then on
    all host threads (at most 16) over the seeded parity subset; the GPU results of the
    parity subset are compared with it element by element."""
    import oracle
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from parity import compare
    h = {k: getattr(w, k).cpu().numpy() for k in
         ("vectors", "ids", "list_offsets", "centroids", "exclude_ids")}
    nq = spec.nq
    rng = np.random.default_rng(spec.seed + 77)
    m1 = min(args.oracle_queries or ORACLE_ONE_THREAD.get(name, 1000), nq)
    sel1 = np.sort(rng.choice(nq, m1, replace=False))
    q1 = w.queries[np.asarray(sel1)].cpu().numpy()
    log(f"[bench] {name}: oracle on {m1} queries, 1 thread")
    t0 = time.perf_counter()
    oracle.search(h["vectors"], h["list_offsets"], h["ids"], h["centroids"], q1,
                  h["exclude_ids"][sel1], spec.k, spec.tau, spec.W, spec.nprobe_max,
                  oracle.MODE_A, 1)
    t1 = time.perf_counter() - t0
    mp = min(ORACLE_PARITY.get(name, 1000), nq)
    selp = np.sort(np.random.default_rng(spec.seed + 501).choice(nq, mp, replace=False))
    qp = w.queries[np.asarray(selp)].cpu().numpy()
    nth = max(1, min(ORACLE_MAX_THREADS, os.cpu_count() or 1))
    log(f"[bench] {name}: oracle on {mp} queries, {nth} threads")
    t0 = time.perf_counter()
    o = oracle.search(h["vectors"], h["list_offsets"], h["ids"], h["centroids"], qp,
                      h["exclude_ids"][selp], spec.k, spec.tau, spec.W, spec.nprobe_max,
                      oracle.MODE_A, nth)
    tp = time.perf_counter() - t0
    rep = compare(ids[selp], scores[selp], probes[selp], o)
    return {
        "cpu_baseline": {"value": round(m1 / t1, 2), "unit": "queries/s", "cores": 1,
                         "kind": "oracle",
                         "sample": f"{m1} seeded queries of the same workload, one thread, "
                                   f"{t1:.1f}s",
                         "threaded": {"value": round(mp / tp, 2), "cores": nth,
                                      "sample": f"the {mp}-query parity subset, {nth} "
                                                f"threads over disjoint query blocks, "
                                                f"{tp:.1f}s"},
                         "cpu": _cpu_model()},
        "parity_sample": {k: rep[k] for k in ("queries", "mismatch", "flag_tau_edge",
                                              "flag_kth_tie", "flag_order_tie",
                                              "flagged_mismatch", "max_score_err")}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="all",
                    help="all (every workload, the 100M one as the headline) or one of "
                         "c1, c2, c3, c5")
    ap.add_argument("--oracle-queries", type=int, default=None,
                    help="queries in the single-thread oracle sample (default: about 5-15 s "
                         "of oracle work for the workload)")
    ap.add_argument("--no-oracle", action="store_true")
    ap.add_argument("--skip-calibrated", action="store_true",
                    help="do not time the in-call calibrated search (profiling runs)")
    ap.add_argument("--sieve-only", action="store_true",
                    help="time the threshold-search steps only (no speculative, fixed-probe, "
                         "calibrated or oracle legs): for counter runs")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 1 GiB device copy (HBM counter calibration)")
    ap.add_argument("--envelope", action="store_true",
                    help="k in {5, 10, 20, 50} and tau in {0.10 .. 0.90} on the 1M x 128 data: "
                         "queries/s, speedup over fixed probing, candidates, overlap with the "
                         "fixed-probe output (one JSON line)")
    ap.add_argument("--concurrency", action="store_true",
                    help="queries per call in {1, 10, 100, 1000, 10000} on the 1M x 128 data, "
                         "for Algorithm 2 lookahead (with and without speculative issue), "
                         "basic and serial dispatch and fixed probing (one JSON line)")
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
        print("bench.py: this build measures one GPU; every box here has one GPU, so --gpus "
              "must be 1 (the multi-GPU design is described, not built)", file=sys.stderr)
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
    names = CONFIG_ORDER if args.config == "all" else [args.config]
    head = "c5" if "c5" in names else names[-1]
    results = {}
    for name in names:
        results[name] = run_config(name, args, ps, sw, np, torch, dev, name == head)
        log(f"[bench] {name}: {json.dumps({k: results[name].get(k) for k in ('qps', 'speedup_vs_fixed', 'rounds', 'mean_probes')})}")
    hr = results[head]
    spec = sw.SPECS[head]
    out = {
        "metric": "queries/sec at W=8 (k=10, tau); speedup vs fixed-nprobe; scan HBM GB/s",
        "value": hr["qps"],
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": hr["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic (seeded mixture + near-duplicate groups, spherical k-means IVF)",
        "config": {"workload": hr["workload"], "queries": spec.nq, "k": spec.k,
                   "tau": spec.tau, "W": spec.W, "nprobe_max": spec.nprobe_max,
                   "fixed_nprobe": spec.fixed_nprobe, "lookahead": "Algorithm 2 (committed)",
                   "parallelism": "single GPU"},
        "speedup_vs_fixed": hr.get("speedup_vs_fixed"),
        "fixed_qps": hr.get("fixed_qps"),
        "partition_vectors_per_s": hr["partition_vectors_per_s"],
        "scan_hbm_gbs": hr["scan_hbm_gbs"],
        "mean_probes": hr["mean_probes"],
        "scanned_probes_per_query": hr["scanned_probes_per_query"],
        "rounds": hr["rounds"],
        "phase_ms": hr["phase_ms"],
        "fixed_phase_ms": hr.get("fixed_phase_ms"),
        "roofline": hr["roofline"],
        "speculative": hr.get("speculative"),
        "calibrated": hr.get("calibrated"),
        "e1": hr["e1"],
        "lists": hr["lists"],
        "paper_context": "4.1-7.6x over fixed probing on 10M workloads and 6.1-8.4x on 100M "
                         "workloads at W=8, 32-core EPYC 7K62 CPU, RaBitQ-coded Lance "
                         "indexes (context only)",
        "configs": {n: results[n] for n in names if n != head},
    }
    if "cpu_baseline" in hr:
        out["cpu_baseline"] = hr["cpu_baseline"]
        out["parity_sample"] = hr["parity_sample"]
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
    Algorithm 2 lookahead with and without speculative issue, basic (Algorithm 1) and serial
    dispatch.  Each point issues consecutive calls
    over a prefix of the 10,000-query batch (at most 200 calls) and reports queries/s."""
    spec = sw.SPECS["c2"]
    log("[concurrency] generating c2")
    w = sw.make(spec, device=dev)
    ix = ps.Index(w.vectors, w.list_offsets, w.ids, w.centroids)
    rows = []
    for per in (1, 10, 100, 1000, 10000):
        calls = min(200, spec.nq // per)
        row = {"queries_per_call": per, "calls": calls}
        for name, kw in (("lookahead", dict(lookahead=True)),
                         ("speculative", dict(lookahead=True, speculative=True)),
                         ("basic", dict(lookahead=False)), ("serial", dict(serial=True)),
                         ("fixed", None)):
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
        row["speculative_vs_fixed"] = round(row["speculative_qps"] / row["fixed_qps"], 3)
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
