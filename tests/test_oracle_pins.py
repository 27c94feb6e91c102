"""Pins for the CPU oracle: checks against what the paper and mathematics fix.

None of these re-types the oracle's own code.  They compare it with
independent numpy brute force (a library matmul plus lexsort), with the stop
rule's closed form and its replay form, with the paper's worked examples
(tests/golden), with the lookahead equivalence argument (Sec. 4.3), with the
prefix property that calibration relies on (Appendix A), and with the
binary16 format itself.  A mutation test then plants plausible mistakes in a
copy of the oracle and checks that some pin fails for each.
"""
import json
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
import sieve_workloads as sw
from sieve_workloads.metrics import pooled_recall

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- helpers
def _np_f64(a):
    return np.asarray(a).astype(np.float64)


def np_order(C, q):
    """Centroid order by (score desc, index asc) from numpy float64."""
    s = _np_f64(C) @ _np_f64(q)
    return np.lexsort((np.arange(len(s)), -s)), s


def np_filtered_topk(X, ids, q, excl, tau, k, rows=None):
    """Exact filtered top-k by numpy float64 (score desc, id asc)."""
    if rows is None:
        rows = np.arange(X.shape[0])
    s = _np_f64(X[rows]) @ _np_f64(q)
    rid = ids[rows]
    keep = (s >= np.float64(np.float32(tau))) & (rid != excl)
    s, rid = s[keep], rid[keep]
    o = np.lexsort((rid, -s))[:k]
    out_ids = np.full(k, -1, np.int64)
    out_s = np.full(k, -np.inf)
    out_ids[: len(o)] = rid[o]
    out_s[: len(o)] = s[o]
    return out_ids, out_s, len(s)


def np_hit_sequence(w, q, excl, tau, order):
    """h[j] = 1 iff the list at rank j+1 holds a non-excluded row with score >= tau."""
    X, ids, off = w["vectors"], w["ids"], w["list_offsets"]
    h = np.zeros(len(order), np.uint8)
    for j, p in enumerate(order):
        rows = np.arange(off[p], off[p + 1])
        if rows.size == 0:
            continue
        s = _np_f64(X[rows]) @ _np_f64(q)
        ok = (s >= np.float64(np.float32(tau))) & (ids[rows] != excl)
        h[j] = 1 if ok.any() else 0
    return h


def replay_probes(h, W):
    """First rank at which W consecutive empties have completed, else len(h)."""
    run = 0
    for j, x in enumerate(h, start=1):
        run = 0 if x else run + 1
        if run >= W:
            return j
    return len(h)


def closed_form_probes(h, W, probes):
    """min(L + W, n) with L the last hit rank inside the visited prefix (0 if none)."""
    n = len(h)
    hits = [j for j in range(1, probes + 1) if h[j - 1]]
    L = hits[-1] if hits else 0
    return min(L + W, n)


def run(w, **kw):
    args = dict(k=10, tau=0.9, W=3, nprobe_max=12, mode=oracle.MODE_A)
    args.update(kw)
    return oracle.search(w["vectors"], w["list_offsets"], w["ids"], w["centroids"], w["queries"],
                         w["exclude_ids"], args["k"], args["tau"], args["W"], args["nprobe_max"],
                         args["mode"], want_hitseq=True, want_order=True)


@pytest.fixture(scope="module")
def tiny(oracle_lib):
    return sw.make("tiny", device="cpu").numpy()


@pytest.fixture(scope="module")
def tiny16(oracle_lib):
    return sw.make("tiny16", device="cpu").numpy()


def random_index(seed, n=600, d=16, nlist=8, nq=40, dtype=np.float32, empty_lists=0):
    """Unstructured random index (lists need not be nearest-centroid: search must not care)."""
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d))
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    # plant near-duplicates so that hits exist
    X[1::7] = X[0::7][: len(X[1::7])] + 0.05 * rng.standard_normal((len(X[1::7]), d))
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    C = rng.standard_normal((nlist, d))
    C /= np.linalg.norm(C, axis=1, keepdims=True)
    sizes = rng.multinomial(n, np.ones(nlist) / nlist)
    if empty_lists:
        sizes[1:1 + empty_lists] = 0
        sizes[0] += n - sizes.sum()
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    ids = rng.permutation(n).astype(np.int64) + 100
    qrows = rng.choice(n, nq, replace=False)
    return {"vectors": X.astype(dtype), "ids": ids, "list_offsets": off,
            "centroids": C.astype(dtype), "queries": X[qrows].astype(dtype),
            "exclude_ids": ids[qrows]}


# ---------------------------------------------------------------- pins
def test_half_decoder_matches_ieee_binary16(oracle_lib):
    bits = np.arange(65536, dtype=np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([oracle.half_to_double(int(b)) for b in bits[::1]])
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(got))
    assert np.array_equal(ref[~nan], got[~nan])


@pytest.mark.parametrize("name", ["tiny", "tiny16"])
def test_rank_order_matches_numpy(name, request):
    w = request.getfixturevalue(name)
    r = run(w, nprobe_max=16)
    for i in range(len(w["queries"])):
        o, s = np_order(w["centroids"], w["queries"][i])
        o = o[: r.order.shape[1]]
        if not np.array_equal(o, r.order[i]):
            # only acceptable where numpy's summation order can flip an exact tie
            ss = np.sort(s)[::-1]
            assert np.min(np.diff(ss[: len(o) + 1]) * -1) < 1e-12, i


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_full_probe_equals_exact_filtered_topk(seed, oracle_lib):
    w = random_index(seed, empty_lists=seed)
    nlist = w["centroids"].shape[0]
    for mode in (oracle.MODE_A, oracle.MODE_B):
        r = run(w, W=oracle.W_INF, nprobe_max=nlist, tau=0.8, k=7, mode=mode)
        bf = oracle.bruteforce(w["vectors"], w["ids"], w["queries"], w["exclude_ids"], 7, 0.8)
        for i in range(len(w["queries"])):
            ei, es, cnt = np_filtered_topk(w["vectors"], w["ids"], w["queries"][i],
                                           w["exclude_ids"][i], 0.8, 7)
            assert np.array_equal(r.ids[i], ei)
            assert np.array_equal(bf.ids[i], ei)
            fin = np.isfinite(es)
            assert np.allclose(r.scores[i][fin], es[fin], atol=1e-12, rtol=0)
            assert np.all(~np.isfinite(r.scores[i][~fin]))
            assert r.ncand[i] == cnt == bf.count[i]
            assert r.probes[i] == nlist


def _shard(w, parts, seed):
    """Split an index's rows into `parts` independently built indexes (same centroids, each
    row kept in its list), ids unchanged."""
    rng = np.random.default_rng(seed)
    owner = rng.integers(0, parts, len(w["ids"]))
    off = np.asarray(w["list_offsets"])
    lists = np.repeat(np.arange(len(off) - 1), np.diff(off))
    out = []
    for p in range(parts):
        rows = np.nonzero(owner == p)[0]  # ascending: lists stay contiguous and in order
        cnt = np.bincount(lists[rows], minlength=len(off) - 1)
        out.append({"vectors": np.ascontiguousarray(w["vectors"][rows]),
                    "ids": np.ascontiguousarray(w["ids"][rows]),
                    "list_offsets": np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64),
                    "centroids": w["centroids"]})
    return out


@pytest.mark.parametrize("seed", [0, 1])
def test_multi_index_full_probe_equals_exact_filtered_topk(seed, oracle_lib):
    """Multi-index search (Sec. 6.1's shards): with no early stop and every list probed in
    every shard, the merged result is the exact filtered top-k over the union of the shards,
    and probes add up over the shards."""
    w = random_index(seed, empty_lists=0)
    nlist = w["centroids"].shape[0]
    shards = _shard(w, 3, seed)
    r = oracle.search_multi(shards, w["queries"], w["exclude_ids"], 7, 0.8, oracle.W_INF, nlist)
    for i in range(len(w["queries"])):
        ei, es, _ = np_filtered_topk(w["vectors"], w["ids"], w["queries"][i],
                                     w["exclude_ids"][i], 0.8, 7)
        assert np.array_equal(r.ids[i], ei)
        fin = np.isfinite(es)
        assert np.allclose(r.scores[i][fin], es[fin], atol=1e-12, rtol=0)
        assert r.probes[i] == 3 * nlist


def test_multi_index_keeps_each_shards_stop_rule(tiny):
    """Each shard stops on its own: the merged probes are the sum of the shards' searches
    run alone, and one shard alone gives its own result back."""
    shards = _shard(tiny, 2, 5)
    args = (tiny["queries"], tiny["exclude_ids"], 10, 0.9, 3, 12)
    r = oracle.search_multi(shards, *args)
    alone = [oracle.search(sh["vectors"], sh["list_offsets"], sh["ids"], sh["centroids"], *args)
             for sh in shards]
    assert np.array_equal(r.probes, alone[0].probes + alone[1].probes)
    one = oracle.search_multi(shards[:1], *args)
    assert np.array_equal(one.ids, alone[0].ids)


@pytest.mark.parametrize("W", [1, 2, 3, 5, 12])
def test_probes_match_replay_and_closed_form(tiny, W):
    r = run(tiny, W=W, nprobe_max=12)
    for i in range(len(tiny["queries"])):
        o, _ = np_order(tiny["centroids"], tiny["queries"][i])
        h = np_hit_sequence(tiny, tiny["queries"][i], tiny["exclude_ids"][i], 0.9, o[:12])
        p = replay_probes(h, W)
        assert r.probes[i] == p, (i, h, W)
        assert r.probes[i] == closed_form_probes(h, W, p)
        # the oracle's own recorded outcomes agree with numpy on the visited prefix
        assert np.array_equal(r.hitseq[i][:p], h[:p])
        assert np.all(r.hitseq[i][p:] == 2)
        hits = np.nonzero(h[:p])[0]
        assert r.last_hit[i] == (hits[-1] + 1 if hits.size else 0)


@pytest.mark.parametrize("name", ["tiny", "tiny16"])
@pytest.mark.parametrize("W", [1, 2, 3, 4, 7, oracle.W_INF])
def test_lookahead_equivalence_mode_a_equals_mode_b(name, W, request):
    w = request.getfixturevalue(name)
    a = run(w, W=W, mode=oracle.MODE_A)
    b = run(w, W=W, mode=oracle.MODE_B)
    for key in ("ids", "scores", "probes", "last_hit", "hitseq", "scanned", "ncand", "rank"):
        assert np.array_equal(a[key], b[key]), key


def test_large_window_equals_fixed_probe(tiny):
    f = oracle.search_fixed(tiny["vectors"], tiny["list_offsets"], tiny["ids"], tiny["centroids"],
                            tiny["queries"], tiny["exclude_ids"], 10, 0.9, 12)
    for W in (12, 13, 1000, oracle.W_INF):
        a = run(tiny, W=W, nprobe_max=12)
        assert np.array_equal(a.ids, f.ids) and np.array_equal(a.scores, f.scores)
        assert np.all(a.probes == 12) and np.all(f.probes == 12)


def test_nprobe_clamped_to_nlist(tiny):
    a = run(tiny, W=oracle.W_INF, nprobe_max=10_000)
    assert np.all(a.probes == tiny["centroids"].shape[0])


@pytest.mark.parametrize("W", [1, 2, 3, 5])
def test_prefix_property(tiny, W):
    """Appendix A: every fixed-probe neighbour found inside W's prefix is kept by W."""
    f = run(tiny, W=oracle.W_INF, nprobe_max=12)
    a = run(tiny, W=W, nprobe_max=12)
    for i in range(len(tiny["queries"])):
        inside = {int(x) for x, rk in zip(f.ids[i], f.rank[i]) if x >= 0 and rk <= a.probes[i]}
        assert inside <= {int(x) for x in a.ids[i] if x >= 0}


def test_self_exclusion(tiny):
    with_ex = run(tiny, W=3)
    no_ex = oracle.search(tiny["vectors"], tiny["list_offsets"], tiny["ids"], tiny["centroids"],
                          tiny["queries"], None, 10, 0.9, 3, 12)
    for i in range(len(tiny["queries"])):
        me = tiny["exclude_ids"][i]
        assert me not in set(with_ex.ids[i].tolist())
        assert no_ex.ids[i][0] == me or np.isclose(no_ex.scores[i][0], 1.0, atol=1e-5)
        assert me in set(no_ex.ids[i].tolist())


def test_exact_assignment_on_generated_index(tiny):
    off = tiny["list_offsets"]
    row_list = np.empty(tiny["vectors"].shape[0], np.int64)
    for c in range(len(off) - 1):
        row_list[tiny["ids"][off[c]:off[c + 1]]] = c
    r = run(tiny, nprobe_max=1, W=1)
    assert np.array_equal(r.order[:, 0], row_list[tiny["exclude_ids"]])


# ------------------------------------------------------- worked examples
def _hand_index(hits, nprobe, tau=0.9):
    """One query q = e0; list j (0-based) is probed at rank j+1 by construction.

    Centroid j = normalize(cos(a_j) e0 + sin(a_j) e1) with a_j increasing,
    so <q, c_j> strictly decreases with j.  A hit list holds a row close to
    e0; every list also holds a row orthogonal to e0.
    """
    d, nlist = 8, nprobe
    ang = np.linspace(0.1, 1.4, nlist)
    C = np.zeros((nlist, d), np.float32)
    C[:, 0], C[:, 1] = np.cos(ang), np.sin(ang)
    rows, ids, off = [], [], [0]
    for j in range(nlist):
        far = np.zeros(d)
        far[2] = far[3] = np.sqrt(0.5)
        rows.append(far)
        if (j + 1) in hits:
            near = np.zeros(d)
            near[0], near[4] = 1.0, 0.05
            rows.append(near / np.linalg.norm(near))
        off.append(len(rows))
    X = np.array(rows, np.float32)
    q = np.zeros((1, d), np.float32)
    q[0, 0] = 1.0
    return {"vectors": X, "ids": np.arange(len(rows), dtype=np.int64) + 10,
            "list_offsets": np.array(off, np.int64), "centroids": C, "queries": q,
            "exclude_ids": np.array([-5], np.int64)}


def test_golden_stop_rule_examples(oracle_lib):
    with open(os.path.join(GOLDEN, "stop_rule_examples.json")) as f:
        cases = json.load(f)["cases"]
    assert len(cases) >= 5
    for c in cases:
        w = _hand_index(set(c["hits"]), c["nprobe"])
        for mode in (oracle.MODE_A, oracle.MODE_B):
            r = run(w, W=c["W"], nprobe_max=c["nprobe"], mode=mode, k=4)
            assert r.probes[0] == c["probes"], (c["name"], mode, r.probes[0])


def test_threshold_is_inclusive(oracle_lib):
    """Sec. 2.2 defines R(q, tau) with >=: a score exactly equal to tau qualifies."""
    tau = np.float32(0.90625)  # exactly representable, so the dot product is exact
    d = 8
    x = np.zeros((3, d), np.float32)
    x[0, 0], x[0, 1] = tau, np.float32(np.sqrt(1 - float(tau) ** 2))
    x[1, 2] = 1.0
    x[2, 0] = np.float32(0.5)
    q = np.zeros((1, d), np.float32)
    q[0, 0] = 1.0
    C = np.eye(d, dtype=np.float32)[:1]
    w = {"vectors": x, "ids": np.array([5, 6, 7], np.int64), "list_offsets": np.array([0, 3]),
         "centroids": C, "queries": q, "exclude_ids": np.array([-1], np.int64)}
    r = run(w, tau=float(tau), W=1, nprobe_max=1, k=2)
    assert r.ids[0][0] == 5 and r.scores[0][0] == float(tau) and r.ids[0][1] == -1


def test_exact_score_ties_break_by_id(oracle_lib):
    d = 8
    x = np.zeros((4, d), np.float32)
    x[:, 0] = 1.0  # four identical rows, identical scores
    q = np.zeros((1, d), np.float32)
    q[0, 0] = 1.0
    C = np.zeros((3, d), np.float32)
    C[:, 0] = 1.0  # identical centroids: order by index
    w = {"vectors": x, "ids": np.array([40, 10, 30, 20], np.int64),
         "list_offsets": np.array([0, 0, 4, 4]), "centroids": C, "queries": q,
         "exclude_ids": np.array([30], np.int64)}
    r = run(w, tau=0.5, W=2, nprobe_max=3, k=3)
    assert r.order[0].tolist() == [0, 1, 2]
    assert r.ids[0].tolist() == [10, 20, 40]
    # list 0 is empty (an empty probe), list 1 hits, list 2 is empty: probes = min(2 + 2, 3)
    assert r.probes[0] == 3 and r.hitseq[0].tolist() == [0, 1, 0]


# ------------------------------------------------------------------ flags
# The flags mark the queries whose outcome a lower-precision implementation may
# legitimately decide the other way (the parity bar excuses mismatches only
# there): TAU_EDGE when a scanned, non-excluded score in a visited list lies
# within 1e-4 of tau; KTH_TIE when the best candidate left out of the top-k lies
# within 1e-4 of the k-th; ORDER_TIE when two returned neighbours lie within
# 1e-4 of each other.  Scores are placed exactly by construction: the query is
# e0 and a row (a, sqrt(1 - a^2), 0, ...) scores a.
BAND = 1e-4


def _ladder_index(scores, ids=None, exclude=-1, far_list_scores=()):
    """One query q = e0.  List 0 (ranked first) holds rows scoring exactly the
    given fp32 values; list 1 (ranked second, never visited with nprobe 1)
    holds rows scoring far_list_scores."""
    d = 8
    rows = []
    for a in list(scores) + list(far_list_scores):
        a = float(np.float32(a))
        x = np.zeros(d)
        x[0] = a
        x[1] = np.sqrt(max(0.0, 1.0 - a * a))
        rows.append(x)
    X = np.array(rows, np.float32) if rows else np.zeros((0, d), np.float32)
    # the score is X[:, 0] exactly: q has a single non-zero, 1.0, in dimension 0
    C = np.zeros((2, d), np.float32)
    C[0, 0], C[0, 2] = 0.9, np.sqrt(1 - 0.81)
    C[1, 0], C[1, 2] = 0.5, np.sqrt(1 - 0.25)
    q = np.zeros((1, d), np.float32)
    q[0, 0] = 1.0
    n0 = len(scores)
    ids = np.arange(len(rows), dtype=np.int64) + 100 if ids is None else np.asarray(ids, np.int64)
    return {"vectors": X, "ids": ids, "list_offsets": np.array([0, n0, len(rows)], np.int64),
            "centroids": C, "queries": q, "exclude_ids": np.array([exclude], np.int64)}


def _flags(w, tau, k=3, nprobe=1, W=1):
    r = run(w, tau=tau, k=k, W=W, nprobe_max=nprobe)
    f = int(r.flags[0])
    return (bool(f & oracle.FLAG_TAU_EDGE), bool(f & oracle.FLAG_KTH_TIE),
            bool(f & oracle.FLAG_ORDER_TIE))


def test_flag_tau_edge_band(oracle_lib):
    tau = float(np.float32(0.9))
    far = [0.1]
    for off, want in ((5e-5, True), (-5e-5, True), (0.0, True), (2e-4, False), (-2e-4, False),
                      (3e-3, False)):
        w = _ladder_index([0.2, tau + off], far_list_scores=far)
        assert _flags(w, tau)[0] == want, off
    # the query's own row is never scanned, so it never flags
    w = _ladder_index([0.2, tau + 1e-5], ids=[100, 101, 102], exclude=101, far_list_scores=far)
    assert _flags(w, tau)[0] is False
    # a list the stop rule never visits never flags
    w = _ladder_index([0.2, 0.3], far_list_scores=[tau + 1e-5])
    assert _flags(w, tau, nprobe=1)[0] is False
    assert _flags(w, tau, nprobe=2, W=5)[0] is True


def test_flag_kth_tie_band(oracle_lib):
    tau = 0.5
    base = [0.99, 0.98, 0.97]  # k = 3 returned
    for gap, want in ((5e-5, True), (0.0, True), (2e-4, False), (1e-3, False)):
        w = _ladder_index(base + [0.97 - gap, 0.6])
        assert _flags(w, tau, k=3)[1] == want, gap
    # no (k+1)-th candidate: nothing can take the k-th slot
    assert _flags(_ladder_index(base), tau, k=3)[1] is False
    # a near tie below the boundary ((k+1)-th vs (k+2)-th) is not a k-th tie
    w = _ladder_index(base + [0.90, 0.90 - 1e-5])
    assert _flags(w, tau, k=3)[1] is False
    # a near tie above it (1st vs (k+1)-th within the band only through the k-th) is not either
    w = _ladder_index([0.99, 0.99 - 5e-5, 0.95, 0.80])
    assert _flags(w, tau, k=3)[1] is False
    # candidates below tau do not count as the (k+1)-th
    w = _ladder_index(base + [0.97 - 5e-5])
    assert _flags(w, 0.97 - 1e-3 + 0.0, k=3)[1] is True
    assert _flags(w, float(np.float32(0.97)) + 0.0, k=3)[1] is False


def test_flag_order_tie_band(oracle_lib):
    tau = 0.5
    for gap, want in ((5e-5, True), (0.0, True), (2e-4, False)):
        w = _ladder_index([0.99, 0.95, 0.95 - gap, 0.7])
        assert _flags(w, tau, k=3)[2] == want, gap
    # only returned neighbours count: a tie between the k-th and the (k+1)-th
    # is a k-th tie, not an order tie
    w = _ladder_index([0.99, 0.95, 0.90, 0.90 - 5e-5])
    assert _flags(w, tau, k=3) == (False, True, False)
    # the first and the last returned pair are both inspected
    w = _ladder_index([0.99, 0.99 - 5e-5, 0.90, 0.80])
    assert _flags(w, tau, k=3)[2] is True
    w = _ladder_index([0.99, 0.90, 0.80, 0.80 - 5e-5, 0.6])
    assert _flags(w, tau, k=4)[2] is True


def _np_flags_one(w, i, tau, k, W, n, order):
    """Flags of query i from numpy float64 scores over the visited prefix (numpy order,
    numpy hit sequence, replayed stop rule): (tau_edge, kth_tie, order_tie, candidates)."""
    X, ids, off = w["vectors"], w["ids"], w["list_offsets"]
    q, ex = w["queries"][i], w["exclude_ids"][i]
    t = np.float64(np.float32(tau))
    h = np_hit_sequence(w, q, ex, tau, order[:n])
    p = replay_probes(h, W)
    edge = False
    cand = []
    for j in range(p):
        rows = np.arange(off[order[j]], off[order[j] + 1])
        rows = rows[ids[rows] != ex]
        s = _np_f64(X[rows]) @ _np_f64(q)
        edge |= bool(np.any(np.abs(s - t) < BAND))
        cand += [(float(v), int(x)) for v, x in zip(s, ids[rows]) if v >= t]
    cand.sort(key=lambda c: (-c[0], c[1]))
    kth = len(cand) > k and cand[k - 1][0] - cand[k][0] < BAND
    top = cand[:k]
    otie = any(top[j][0] - top[j + 1][0] < BAND for j in range(len(top) - 1))
    return edge, kth, otie, cand


def _flag_rich_index(seed, tau):
    """A random index with score ladders planted around tau and around each query's
    top candidates, so that every flag is set for some queries and clear for others."""
    rng = np.random.default_rng(seed)
    w = random_index(seed, n=500, d=16, nlist=6, nq=24)
    X = w["vectors"].astype(np.float64)
    extra = []
    for qv in w["queries"].astype(np.float64):
        qn = qv / np.linalg.norm(qv)
        for _ in range(4):
            # a row scoring tau + u (|u| up to 3e-4) and a pair 0 .. 2e-4 apart near 0.97
            for a in (tau + rng.uniform(-3e-4, 3e-4), 0.97, 0.97 - rng.uniform(0, 2e-4)):
                u = rng.standard_normal(X.shape[1])
                u -= (u @ qn) * qn
                u /= np.linalg.norm(u)
                extra.append(a * qn + np.sqrt(1 - a * a) * u)
    E = np.array(extra)
    Xa = np.concatenate([X, E]).astype(np.float32)
    # every planted row joins its nearest centroid's list (row order by list)
    C = w["centroids"].astype(np.float64)
    lst = np.argmax(Xa.astype(np.float64) @ C.T, axis=1)
    o = np.argsort(lst, kind="stable")
    ids = np.arange(len(Xa), dtype=np.int64)[o] + 7
    qrows = rng.choice(len(X), len(w["queries"]), replace=False)
    Xs = Xa[o]
    pos = np.empty(len(o), np.int64)
    pos[o] = np.arange(len(o))
    return {"vectors": Xs, "ids": ids,
            "list_offsets": np.concatenate([[0], np.cumsum(np.bincount(lst, minlength=len(C)))]
                                           ).astype(np.int64),
            "centroids": w["centroids"], "queries": Xa[qrows], "exclude_ids": qrows + 7}


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_flags_match_numpy_on_random_indexes(seed, oracle_lib):
    """Every flag bit, recomputed from numpy float64 scores over the visited prefix."""
    tau = 0.6
    w = _flag_rich_index(seed, tau)
    nlist = w["centroids"].shape[0]
    seen = np.zeros(3, int)
    for W, k, npb in ((1, 3, nlist), (2, 5, 4), (oracle.W_INF, 4, nlist)):
        r = run(w, tau=tau, k=k, W=W, nprobe_max=npb)
        n = min(npb, nlist)
        for i in range(len(w["queries"])):
            order, _ = np_order(w["centroids"], w["queries"][i])
            edge, kth, otie, _ = _np_flags_one(w, i, tau, k, W, n, order)
            f = int(r.flags[i])
            got = (bool(f & oracle.FLAG_TAU_EDGE), bool(f & oracle.FLAG_KTH_TIE),
                   bool(f & oracle.FLAG_ORDER_TIE))
            assert got == (edge, kth, otie), (seed, W, k, i)
            seen += np.array(got, int)
    # the planted ladders make every flag occur (and not everywhere)
    total = 3 * len(w["queries"])
    assert np.all(seen > 0) and np.all(seen < total), seen


def test_multi_index_flags_match_numpy(oracle_lib):
    """search_multi's flags: TAU_EDGE of any shard (each shard's own visited lists);
    KTH_TIE of any shard or at the boundary of the merged candidates; ORDER_TIE among
    the merged top-k."""
    tau, k, W = 0.6, 4, 1
    w = _flag_rich_index(5, tau)
    nlist = w["centroids"].shape[0]
    shards = _shard(w, 3, 11)
    r = oracle.search_multi(shards, w["queries"], w["exclude_ids"], k, tau, W, nlist)
    seen = np.zeros(3, int)
    for i in range(len(w["queries"])):
        edge = kth = False
        allc = []
        for sh in shards:
            sh_w = dict(sh, queries=w["queries"], exclude_ids=w["exclude_ids"])
            order, _ = np_order(sh["centroids"], w["queries"][i])
            e, kt, _, c = _np_flags_one(sh_w, i, tau, k, W, nlist, order)
            edge |= e
            kth |= kt
            allc += c
        allc.sort(key=lambda c: (-c[0], c[1]))
        kth |= len(allc) > k and allc[k - 1][0] - allc[k][0] < BAND
        top = allc[:k]
        otie = any(top[j][0] - top[j + 1][0] < BAND for j in range(len(top) - 1))
        f = int(r.flags[i])
        got = (bool(f & oracle.FLAG_TAU_EDGE), bool(f & oracle.FLAG_KTH_TIE),
               bool(f & oracle.FLAG_ORDER_TIE))
        assert got == (edge, kth, otie), i
        assert [x for x in r.ids[i] if x >= 0] == [c[1] for c in top]
        seen += np.array(got, int)
    assert np.all(seen > 0), seen


# ------------------------------------------------------------ calibration
def test_calibration_replay_matches_direct_runs(tiny):
    """Appendix A: H's prefix sums equal the retained counts of actual W runs."""
    n = 12
    f = run(tiny, W=oracle.W_INF, nprobe_max=n)
    wsel, hist, z = oracle.calibrate(f.hitseq, f.rank, eps=0.005)
    assert z == int((f.ids >= 0).sum())
    fixed_sets = [{int(x) for x in row if x >= 0} for row in f.ids]
    for W in range(1, n):
        a = run(tiny, W=W, nprobe_max=n)
        kept = sum(len(fs & {int(x) for x in row if x >= 0}) for fs, row in zip(fixed_sets, a.ids))
        assert kept == hist[1:W + 1].sum(), W
    # chosen window: smallest W < n with loss < eps, else n
    losses = [1 - hist[1:W + 1].sum() / z for W in range(1, n)]
    want = next((W for W, l in zip(range(1, n), losses) if l < 0.005), n)
    assert wsel == want


def test_calibration_hand_case(oracle_lib):
    # one query, n = 6; hits at ranks 1 and 5; neighbours found at ranks 1 and 5.
    h = np.array([[1, 0, 0, 0, 1, 0]], np.uint8)
    fr = np.array([[1, 5, 0]], np.int32)
    # rank 1 is reached by every W (required window 1); rank 5 needs the
    # empty run 2..4 to stay below W, i.e. W >= 4.
    wsel, hist, z = oracle.calibrate(h, fr, eps=0.5)
    assert z == 2 and hist.tolist() == [0, 1, 0, 0, 1, 0, 0]
    assert wsel == 4  # loss(1..3) = 0.5 is not < 0.5; loss(4) = 0
    wsel, _, _ = oracle.calibrate(h, fr, eps=0.6)
    assert wsel == 1
    wsel, _, z = oracle.calibrate(np.zeros((1, 6), np.uint8), np.zeros((1, 3), np.int32), 0.1)
    assert wsel is None and z == 0


# --------------------------------------------------------------- metrics
def test_pooled_recall_toy():
    # q0: G={1,2,3}, A={1,2,9}; q1: G={} (excluded); q2: G={4}, A={4}
    G = [[1, 2, 3], [-1, -1, -1], [4, -1, -1]]
    A = [[1, 2, 9], [7, -1, -1], [4, -1, -1]]
    r, num, den = pooled_recall(A, G)
    assert (num, den) == (3, 4) and r == 0.75


# -------------------------------------------------------------- mutation
MUTANTS = {
    "no_stale_reset": ("        run = 0;\n        last_hit = j;", "        last_hit = j;"),
    "strict_threshold": ("    if (v >= tau) {", "    if (v > tau) {"),
    "id_tiebreak_reversed": ("  if (a->id < b->id) return -1;\n  if (a->id > b->id) return 1;",
                             "  if (a->id < b->id) return 1;\n  if (a->id > b->id) return -1;"),
    "centroid_tiebreak_reversed": ("  return (a->c > b->c) - (a->c < b->c);",
                                   "  return (a->c < b->c) - (a->c > b->c);"),
    "dropped_last_dim": ("  for (int t = 0; t < d; ++t) s += q[t]",
                         "  for (int t = 0; t < d - 1; ++t) s += q[t]"),
    "no_self_exclusion": ("    if (has_excl && ix->ids[r] == excl) continue;\n    double v",
                          "    double v"),
    "stop_line_short": ("int line = (W > n - j) ? n : j + W;",
                        "int line = (W > n - j) ? n : j + W - 1;"),
    "stop_one_late": ("      } else if (++run >= W) {", "      } else if (++run > W) {"),
    "order_ascending": ("  if (a->s > b->s) return -1;\n  if (a->s < b->s) return 1;\n  return (a->c",
                        "  if (a->s > b->s) return 1;\n  if (a->s < b->s) return -1;\n  return (a->c"),
    # the tie/threshold flags that excuse GPU/oracle differences
    "edge_band_too_wide": ("#define OR_EDGE_BAND 1e-4", "#define OR_EDGE_BAND 1e-2"),
    "tau_edge_always": ("    if (fabs(v - tau) < OR_EDGE_BAND) *flags |= OR_FLAG_TAU_EDGE;",
                        "    *flags |= OR_FLAG_TAU_EDGE;"),
    "tau_edge_counts_excluded": (
        "    if (has_excl && ix->ids[r] == excl) continue;\n"
        "    double v = dot_row(q, ix->vectors, ix->dtype, r, ix->d);\n"
        "    (*scanned)++;\n"
        "    /* a score this close to tau may be decided either way in lower precision */\n"
        "    if (fabs(v - tau) < OR_EDGE_BAND) *flags |= OR_FLAG_TAU_EDGE;\n",
        "    double v = dot_row(q, ix->vectors, ix->dtype, r, ix->d);\n"
        "    if (fabs(v - tau) < OR_EDGE_BAND) *flags |= OR_FLAG_TAU_EDGE;\n"
        "    if (has_excl && ix->ids[r] == excl) continue;\n"
        "    (*scanned)++;\n"),
    "kth_tie_wrong_index": ("cv->v[k - 1].s - cv->v[k].s < OR_EDGE_BAND",
                            "cv->v[0].s - cv->v[k].s < OR_EDGE_BAND"),
    "order_tie_off_by_one": ("  for (int r = 0; r + 1 < kept; ++r)\n    if (cv->v[r].s",
                             "  for (int r = 0; r + 2 < kept; ++r)\n    if (cv->v[r].s"),
}


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_catch_planted_mistakes(mutant, tmp_path, oracle_lib):
    """Plant one plausible mistake in a copy of the oracle; some pin must fail."""
    src = open(os.path.join(os.path.dirname(oracle.__file__), "sieve_oracle.c")).read()
    old, new = MUTANTS[mutant]
    assert src.count(old) == 1, mutant
    pkg = tmp_path / "oracle"
    pkg.mkdir()
    (pkg / "sieve_oracle.c").write_text(src.replace(old, new))
    shutil.copy(oracle.__file__, pkg / "__init__.py")
    subprocess.check_call(["gcc", *oracle.CFLAGS, "-o", str(pkg / "liboracle.so"),
                           str(pkg / "sieve_oracle.c"), "-lm", "-lpthread"])
    code = f"""
import sys; sys.path.insert(0, {str(tmp_path)!r}); sys.path.insert(1, {os.path.dirname(GOLDEN)!r})
sys.path.insert(2, {os.path.dirname(os.path.dirname(GOLDEN))!r})
import oracle
assert oracle.__file__.startswith({str(tmp_path)!r})
import test_oracle_pins as T
import sieve_workloads as sw
tiny = sw.make("tiny", device="cpu").numpy()
checks = [
    lambda: T.test_golden_stop_rule_examples(None),
    lambda: T.test_threshold_is_inclusive(None),
    lambda: T.test_exact_score_ties_break_by_id(None),
    lambda: T.test_self_exclusion(tiny),
    lambda: T.test_full_probe_equals_exact_filtered_topk(0, None),
    lambda: T.test_probes_match_replay_and_closed_form(tiny, 3),
    lambda: T.test_lookahead_equivalence_mode_a_equals_mode_b("tiny", 3, type("R", (), {{"getfixturevalue": lambda s, n: tiny}})()),
    lambda: T.test_rank_order_matches_numpy("tiny", type("R", (), {{"getfixturevalue": lambda s, n: tiny}})()),
    lambda: T.test_flag_tau_edge_band(None),
    lambda: T.test_flag_kth_tie_band(None),
    lambda: T.test_flag_order_tie_band(None),
    lambda: T.test_flags_match_numpy_on_random_indexes(0, None),
]
failed = 0
for c in checks:
    try:
        c()
    except AssertionError:
        failed += 1
print("FAILED_PINS", failed)
"""
    out = subprocess.run(["python", "-c", code], capture_output=True, text=True, timeout=300)
    assert "FAILED_PINS" in out.stdout, out.stderr[-2000:]
    n_failed = int(out.stdout.split("FAILED_PINS")[1].split()[0])
    assert n_failed >= 1, f"mutant {mutant} survived every pin"
