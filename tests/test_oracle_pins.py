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
    "no_stale_reset": ("        stale = 0;\n        last_hit = j;", "        last_hit = j;"),
    "strict_threshold": ("    if (v >= tau) {", "    if (v > tau) {"),
    "id_tiebreak_reversed": ("  if (a->id < b->id) return -1;\n  if (a->id > b->id) return 1;",
                             "  if (a->id < b->id) return 1;\n  if (a->id > b->id) return -1;"),
    "centroid_tiebreak_reversed": ("  return (a->c > b->c) - (a->c < b->c);",
                                   "  return (a->c < b->c) - (a->c > b->c);"),
    "dropped_last_dim": ("  for (int t = 0; t < d; ++t) s += q[t]",
                         "  for (int t = 0; t < d - 1; ++t) s += q[t]"),
    "no_self_exclusion": ("    if (has_excl && ix->ids[r] == excl) continue;\n    double v",
                          "    double v"),
    "stop_line_short": ("int reach = (W > n - j) ? n : j + W;",
                        "int reach = (W > n - j) ? n : j + W - 1;"),
    "stop_one_late": ("      if (!(stale < W && next <= n)) break;",
                      "      if (!(stale <= W && next <= n)) break;"),
    "order_ascending": ("  if (a->s > b->s) return -1;\n  if (a->s < b->s) return 1;\n  return (a->c",
                        "  if (a->s > b->s) return 1;\n  if (a->s < b->s) return -1;\n  return (a->c"),
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
