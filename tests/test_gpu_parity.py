"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Every case runs the library on seeded synthetic inputs and the oracle on the
same arrays, and compares ids and probe counts exactly and scores to 1e-4
(tests/parity.py states the flagged exceptions).  Sizes span many tiles,
ragged query tiles and ragged row blocks; edge cases cover empty input,
k = 1 and k = 64, nprobe = 1 and nprobe > nlist, W = 1 and W = infinity,
empty lists, dimensions that are not a multiple of the MFMA chunk, and a
threshold low enough to overflow the candidate pool.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import sieve_workloads as sw
from parity import assert_parity, compare

pytestmark = pytest.mark.gpu

NTHREADS = min(16, os.cpu_count() or 1)


def _lib():
    import paper_2608_03199_amd as ps
    return ps


@pytest.fixture(scope="module", autouse=True)
def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    _lib().load_library()


class Case:
    """A workload on the GPU, its library index and host copies for the oracle."""

    def __init__(self, w: sw.Workload):
        ps = _lib()
        self.w = w
        self.h = w.numpy()
        self.ix = ps.Index(w.vectors, w.list_offsets, w.ids, w.centroids)

    def gpu(self, k, tau, W, nprobe, lookahead=True, queries=None, exclude=True, fixed=False,
            stats=False, speculative=False):
        q = self.w.queries if queries is None else queries
        ex = self.w.exclude_ids[: q.shape[0]] if exclude else None
        if fixed:
            r = self.ix.search_fixed(q, ex, k, tau, nprobe, with_stats=stats)
        else:
            r = self.ix.search(q, ex, k, tau, W, nprobe, lookahead=lookahead, with_stats=stats,
                               speculative=speculative)
        torch.cuda.synchronize()
        out = [r[0].cpu().numpy(), r[1].cpu().numpy(), r[2].cpu().numpy()]
        if stats:
            out.append(r[3])
        return out

    def oracle(self, k, tau, W, nprobe, nq=None, exclude=True):
        h = self.h
        qs = h["queries"] if nq is None else h["queries"][:nq]
        ex = (h["exclude_ids"][: qs.shape[0]]) if exclude else None
        return oracle.search(h["vectors"], h["list_offsets"], h["ids"], h["centroids"], qs, ex, k,
                             tau, W, nprobe, oracle.MODE_A, NTHREADS)


_cases = {}


def case(name, **kw) -> Case:
    key = (name, tuple(sorted(kw.items())))
    if key not in _cases:
        print(f"[gpu-test] generating workload {name} {kw}", flush=True)
        _cases[key] = Case(sw.make(name, device="cuda", **kw))
    return _cases[key]


def _check(c: Case, k, tau, W, nprobe, lookahead=True, fixed=False, nq=None, exclude=True,
           speculative=False):
    q = c.w.queries if nq is None else c.w.queries[:nq]
    g_ids, g_sc, g_pr = c.gpu(k, tau, W, nprobe, lookahead, queries=q, exclude=exclude,
                              fixed=fixed, speculative=speculative)
    o = c.oracle(k, tau, oracle.W_INF if fixed else W, nprobe, nq=q.shape[0], exclude=exclude)
    rep = compare(g_ids, g_sc, g_pr, o)
    print(f"[gpu-test] k={k} tau={tau} W={W} nprobe={nprobe} la={lookahead} fixed={fixed} "
          f"-> {rep}", flush=True)
    assert_parity(rep)
    return g_ids, g_sc, g_pr, o


@pytest.fixture
def no_speculation():
    """Lookahead is Algorithm 2 (committed ranks only) unless speculative issue is asked
    for, so it searches exactly the (query, partition) pairs the other dispatches search."""
    yield


@pytest.mark.parametrize("name", ["tiny", "tiny16", "c1"])
@pytest.mark.parametrize("lookahead", [True, False])
def test_sieve_matches_oracle(name, lookahead):
    c = case(name)
    s = c.w.spec
    _check(c, s.k, s.tau, s.W, s.nprobe_max, lookahead)


@pytest.mark.parametrize("name", ["tiny", "tiny16", "c1"])
def test_fixed_matches_oracle(name):
    c = case(name)
    s = c.w.spec
    _check(c, s.k, s.tau, oracle.W_INF, s.fixed_nprobe, fixed=True)


@pytest.mark.parametrize("name", ["tiny16", "c1"])
@pytest.mark.parametrize("W", [1, 2, 4, 16])
def test_lookahead_invariance_and_window_sweep(name, W, no_speculation):
    c = case(name)
    s = c.w.spec
    a = c.gpu(s.k, s.tau, W, s.nprobe_max, lookahead=True, stats=True)
    b = c.gpu(s.k, s.tau, W, s.nprobe_max, lookahead=False, stats=True)
    for x, y in zip(a[:3], b[:3]):
        assert np.array_equal(x, y)
    # the same query-partition searches: same items, probes and scanned rows
    assert a[3].items == b[3].items and a[3].vectors_scanned == b[3].vectors_scanned
    assert a[3].probes_total == b[3].probes_total == int(a[2].sum())
    _check(c, s.k, s.tau, W, s.nprobe_max, lookahead=True)


@pytest.fixture(params=["materialised", "fused"])
def rank_path(request):
    """Run a test under each ranking path: materialised screen scores + selection, and the
    fused screen + selection that short prefixes use on large centroid sets (forced here)."""
    old = os.environ.get("SIEVE_RANK_PATH")
    os.environ["SIEVE_RANK_PATH"] = "1" if request.param == "materialised" else "2"
    yield request.param
    if old is None:
        del os.environ["SIEVE_RANK_PATH"]
    else:
        os.environ["SIEVE_RANK_PATH"] = old


@pytest.fixture
def short_rank_prefix():
    """Order only max(1, 2W) ranks up front, so that stop lines pass the ordered prefix and
    the on-demand extension runs."""
    old = os.environ.get("SIEVE_RANK_PREFIX")
    os.environ["SIEVE_RANK_PREFIX"] = "1"
    yield
    if old is None:
        del os.environ["SIEVE_RANK_PREFIX"]
    else:
        os.environ["SIEVE_RANK_PREFIX"] = old


@pytest.mark.parametrize("name", ["tiny", "c1"])
@pytest.mark.parametrize("W", [1, 2, 4])
def test_lazy_rank_extension(name, W, short_rank_prefix, rank_path, no_speculation):
    # tau = 0.5 makes cluster mates qualify in some queries, so stop lines go deep
    c = case(name)
    s = c.w.spec
    tau = 0.5
    a = c.gpu(s.k, tau, W, s.nprobe_max, lookahead=True, stats=True)
    b = c.gpu(s.k, tau, W, s.nprobe_max, lookahead=False, stats=True)
    # some stop line must have passed the 2W-rank prefix for the test to mean anything
    assert int(a[2].max()) > 2 * W
    for x, y in zip(a[:3], b[:3]):
        assert np.array_equal(x, y)
    assert a[3].items == b[3].items and a[3].vectors_scanned == b[3].vectors_scanned
    _check(c, s.k, tau, W, s.nprobe_max, lookahead=True)
    _check(c, s.k, tau, W, s.nprobe_max, lookahead=False)


@pytest.mark.parametrize("name", ["tiny16", "c1"])
@pytest.mark.parametrize("W", [1, 3, 8])
def test_serial_traversal_matches_batched_dispatch(name, W, no_speculation):
    """Serial traversal (Sec. 6.3's ablation baseline: one rank per query per round, no
    partition scan shared between queries) returns exactly what the batched dispatches
    return, and the oracle's result."""
    c = case(name)
    s = c.w.spec
    q, ex = c.w.queries, c.w.exclude_ids
    a = c.ix.search(q, ex, s.k, s.tau, W, s.nprobe_max, lookahead=True, with_stats=True)
    b = c.ix.search(q, ex, s.k, s.tau, W, s.nprobe_max, serial=True, with_stats=True)
    for x, y in zip(a[:3], b[:3]):
        assert torch.equal(x, y)
    # the same (query, partition) searches, each in a tile of its own
    assert a[3].items == b[3].items and a[3].vectors_scanned == b[3].vectors_scanned
    assert b[3].rounds >= a[3].rounds
    o = c.oracle(s.k, s.tau, W, s.nprobe_max)
    rep = compare(b[0].cpu().numpy(), b[1].cpu().numpy(), b[2].cpu().numpy(), o)
    print(f"[gpu-test] serial {name} W={W} rounds {b[3].rounds} vs {a[3].rounds} -> {rep}",
          flush=True)
    assert_parity(rep)


def _with_speculation(on, fn, first_round=0, spec_min=1):
    """Run fn(speculative) with speculative issue on or off, from round first_round on, for
    stop lines that moved at least spec_min ranks (None: the library's default)."""
    keys = ("SIEVE_SPEC_ROUND", "SIEVE_SPEC_MIN")
    old = {k: os.environ.get(k) for k in keys}
    os.environ["SIEVE_SPEC_ROUND"] = str(first_round)
    if spec_min is None:
        os.environ.pop("SIEVE_SPEC_MIN", None)
    else:
        os.environ["SIEVE_SPEC_MIN"] = str(spec_min)
    try:
        return fn(on)
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


@pytest.mark.parametrize("name,tau", [("tiny", 0.9), ("tiny", 0.5), ("tiny16", 0.6),
                                      ("c1", 0.9), ("c1", 0.5), ("c1", 0.3)])
@pytest.mark.parametrize("W", [1, 2, 5, 8])
@pytest.mark.parametrize("first_round,spec_min", [(0, 1), (1, 1), (2, 1), (0, None)])
def test_speculative_issue_matches_committed_issue(name, tau, W, first_round, spec_min):
    """Lookahead with speculative issue (ranks past the stop line scanned early, the stop
    rule replayed over the per-rank hit bitmap, candidates past the final line dropped)
    returns exactly what committed-only issue returns, and the oracle's result; it never
    needs more rounds, and it searches a superset of the pairs.  first_round: the first
    round whose update speculates (the earlier ones issue committed ranks only); spec_min:
    the shortest move of a stop line that speculates (None: the default, W / 2)."""
    c = case(name)
    s = c.w.spec
    q, ex = c.w.queries, c.w.exclude_ids
    run = lambda sp: c.ix.search(q, ex, s.k, tau, W, s.nprobe_max, with_stats=True,
                                 speculative=sp)
    a = _with_speculation(True, run, first_round, spec_min)
    b = _with_speculation(False, run)
    for x, y in zip(a[:3], b[:3]):
        assert torch.equal(x, y)
    assert a[3].probes_total == b[3].probes_total == int(a[2].sum())
    assert a[3].items >= b[3].items
    assert a[3].rounds <= b[3].rounds
    o = c.oracle(s.k, tau, W, s.nprobe_max)
    rep = compare(a[0].cpu().numpy(), a[1].cpu().numpy(), a[2].cpu().numpy(), o)
    print(f"[gpu-test] speculative {name} tau={tau} W={W} from round {first_round}, "
          f"min move {spec_min}: "
          f"rounds {a[3].rounds} vs "
          f"{b[3].rounds}, items {a[3].items} vs {b[3].items} -> {rep}", flush=True)
    assert_parity(rep)


def test_speculative_issue_with_rank_extension(short_rank_prefix):
    """Speculation stops at the ordered prefix; stop lines that pass it extend the order and
    issue only committed ranks beyond it."""
    c = case("c1")
    s = c.w.spec
    q, ex = c.w.queries, c.w.exclude_ids
    for W in (1, 3):
        run = lambda sp: c.ix.search(q, ex, s.k, 0.4, W, s.nprobe_max, with_stats=True,
                                     speculative=sp)
        a = _with_speculation(True, run, 0)
        b = _with_speculation(False, run)
        assert int(a[2].max()) > 2 * W
        for x, y in zip(a[:3], b[:3]):
            assert torch.equal(x, y)
        assert a[3].rounds <= b[3].rounds
        _with_speculation(True, lambda sp: _check(c, s.k, 0.4, W, s.nprobe_max, lookahead=True,
                                                  speculative=sp))


def test_infinite_window_equals_fixed():
    c = case("c1")
    s = c.w.spec
    a = c.gpu(s.k, s.tau, 0x7FFFFFFF, s.nprobe_max)
    f = c.gpu(s.k, s.tau, 0, s.nprobe_max, fixed=True)
    for x, y in zip(a, f):
        assert np.array_equal(x, y)


def test_repeatable():
    c = case("c1")
    s = c.w.spec
    a = c.gpu(s.k, s.tau, s.W, s.nprobe_max)
    b = c.gpu(s.k, s.tau, s.W, s.nprobe_max)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("k", [1, 7, 64])
def test_k_edges(k):
    c = case("tiny")
    _check(c, k, 0.85, 3, 12)
    _check(c, k, 0.85, 3, 12, fixed=True)


@pytest.mark.parametrize("nprobe", [1, 5, 16, 1000])
def test_nprobe_edges(nprobe):
    c = case("tiny")
    _check(c, 10, 0.9, 2, nprobe)
    _check(c, 10, 0.9, 2, nprobe, fixed=True)


def test_ragged_and_small_batches():
    c = case("c1")
    for nq in (1, 15, 17, 129, 333):
        _check(c, 10, 0.9, 8, 32, nq=nq)
    # no exclusion: every query finds itself at rank 1
    g_ids, g_sc, g_pr, o = _check(c, 10, 0.9, 8, 32, nq=64, exclude=False)
    assert np.array_equal(g_ids[:, 0], c.h["exclude_ids"][:64])


def test_empty_query_batch():
    c = case("tiny")
    ids, sc, pr = c.gpu(10, 0.9, 3, 12, queries=c.w.queries[:0])
    assert ids.shape == (0, 10) and pr.shape == (0,)


@pytest.mark.parametrize("d,dtype", [(40, torch.float32), (72, torch.float16),
                                     (96, torch.float32), (256, torch.float16),
                                     (768, torch.float16)])
def test_uncommon_dimensions(d, dtype, rank_path):
    """Dimensions off the compiled fast paths, including partial MFMA chunks, and d = 768
    fp16 (rows streamed in slices of 8 MFMA chunks)."""
    spec = sw.SPECS["tiny"]
    import dataclasses
    sp = dataclasses.replace(spec, name=f"d{d}", d=d, dtype="f16" if dtype == torch.float16
                             else "f32", n=4000, nlist=24, nq=200)
    c = Case(sw.make(sp, device="cuda"))
    _check(c, 10, 0.9, 3, 12)
    _check(c, 10, 0.9, 3, 24, fixed=True)
    if d == 768:
        # the 768-dim scan also has the two-work-groups-per-CU configuration
        os.environ["SIEVE_SCAN_WIDE"] = "2"
        try:
            _check(c, 10, 0.9, 3, 12)
            _check(c, 10, 0.9, 3, 24, fixed=True)
        finally:
            del os.environ["SIEVE_SCAN_WIDE"]


def test_empty_lists_and_unbalanced_index():
    """Lists of length zero are threshold-empty probes; one list holds most rows."""
    rng = np.random.default_rng(5)
    d, nlist, n = 32, 12, 2500
    X = rng.standard_normal((n, d)).astype(np.float32)
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    X[1::5] = X[0::5][: len(X[1::5])] + 0.03 * rng.standard_normal((len(X[1::5]), d))
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    C = rng.standard_normal((nlist, d)).astype(np.float32)
    C /= np.linalg.norm(C, axis=1, keepdims=True)
    sizes = np.array([0, 2000, 0, 0, 100, 100, 0, 100, 100, 50, 50, 0])
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    ids = rng.permutation(n).astype(np.int64)
    qrows = rng.choice(n, 300, replace=False)
    ps = _lib()
    dev = "cuda"
    ix = ps.Index(torch.from_numpy(X).to(dev), torch.from_numpy(off).to(dev),
                  torch.from_numpy(ids).to(dev), torch.from_numpy(C).to(dev))
    Q = X[qrows].copy()
    ex = ids[qrows]
    for W in (1, 3, 0x7FFFFFFF):
        g = ix.search(torch.from_numpy(Q).to(dev), torch.from_numpy(ex).to(dev), 10, 0.9, W, 12)
        o = oracle.search(X, off, ids, C, Q, ex, 10, 0.9, W, 12)
        rep = compare(g[0].cpu().numpy(), g[1].cpu().numpy(), g[2].cpu().numpy(), o)
        assert_parity(rep)


@pytest.mark.parametrize("d,dtype", [(64, np.float16), (128, np.float16), (768, np.float16),
                                     (64, np.float32), (128, np.float32)])
def test_fragment_copy_with_ragged_partitions(d, dtype):
    """Dimensions whose scan and ranking read the fragment-order copies: partitions of 0, 1,
    15, 16, 17, 33 ... rows, so that padding rows sit between most partitions of the vector
    copy, and 17 centroids, so that the centroid copy ends in a partial block (the fused
    ranking path, which reads it, is forced on the second pass).  Search, fixed probing and,
    with the arena off (every tile with candidates takes the exact top-k pass, which reads
    the copy from its overflow records), the oracle's result every way."""
    rng = np.random.default_rng(11 + d)
    sizes = np.array([0, 1, 15, 16, 17, 33, 0, 300, 5, 31, 48, 64, 129, 0, 2, 47, 90])
    n, nlist = int(sizes.sum()), len(sizes)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    X = rng.standard_normal((n, d))
    X[1::4] = X[0::4][: len(X[1::4])] + 0.02 * rng.standard_normal((len(X[1::4]), d))
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    C = rng.standard_normal((nlist, d))
    C /= np.linalg.norm(C, axis=1, keepdims=True)
    X, C = X.astype(dtype), C.astype(dtype)
    ids = rng.permutation(n).astype(np.int64) + 1000
    qrows = rng.choice(n, 200, replace=False)
    Q, ex = X[qrows].copy(), ids[qrows]
    Xo, Co, Qo = X.astype(np.float32), C.astype(np.float32), Q.astype(np.float32)
    ps = _lib()
    dev = "cuda"
    t = lambda a: torch.from_numpy(a).to(dev)
    for arena, rank_path in (("1", None), ("0", "2")):
        os.environ["SIEVE_ARENA"] = arena  # read when a search sizes its workspace
        if rank_path is not None:
            os.environ["SIEVE_RANK_PATH"] = rank_path
        ix = ps.Index(t(X), t(off), t(ids), t(C))
        try:
            for W, fixed in ((2, False), (0x7FFFFFFF, False), (None, True)):
                if fixed:
                    g = ix.search_fixed(t(Q), t(ex), 10, 0.9, 9, with_stats=True)
                else:
                    g = ix.search(t(Q), t(ex), 10, 0.9, W, 9, with_stats=True)
                o = oracle.search(Xo, off, ids, Co, Qo, ex, 10, 0.9,
                                  oracle.W_INF if fixed else W, 9)
                rep = compare(g[0].cpu().numpy(), g[1].cpu().numpy(), g[2].cpu().numpy(), o)
                print(f"[gpu-test] d={d} {np.dtype(dtype).name} arena={arena} "
                      f"rank_path={rank_path} W={W} "
                      f"fixed={fixed} heavy={g[3].heavy_records} -> {rep}", flush=True)
                assert_parity(rep)
                if arena == "0" and g[3].hits > 0:
                    assert g[3].heavy_records > 0
        finally:
            del os.environ["SIEVE_ARENA"]
            os.environ.pop("SIEVE_RANK_PATH", None)
            ix.close()


def test_low_threshold_pool_and_overflow_records_grow():
    """tau = -1: every scanned row qualifies.  With k = 64 and 32 probes per query the
    pool, though bounded by k entries per (query, tile), needs about 2M entries for 1,000
    queries, more than a fresh index's first pool (about 1M), so it grows and the search
    re-runs; with the overflow-record buffer started at 2 records through its knob, that
    buffer grows too (queries whose pairs overflow a tile's arena get records).  A second
    search needs no retry and gives the same result."""
    ps = _lib()
    c = case("c1")
    ix = ps.Index(c.w.vectors, c.w.list_offsets, c.w.ids, c.w.centroids)
    try:
        os.environ["SIEVE_HEAVY_CAP0"] = "2"  # read when the first search sizes the buffer
        try:
            r = ix.search(c.w.queries, c.w.exclude_ids, 64, -1.0, 4, 32, with_stats=True)
        finally:
            del os.environ["SIEVE_HEAVY_CAP0"]
        g_ids, g_sc, g_pr, st = (t.cpu().numpy() if hasattr(t, "cpu") else t for t in r)
        print(f"[gpu-test] tau -1, k 64: retries {st.pool_retries}, found {st.hits}, "
              f"pool {st.pool_entries}, heavy records {st.heavy_records}", flush=True)
        assert st.pool_retries >= 2 and st.heavy_records > 2
        assert st.hits > 8_000_000 and st.pool_entries > (1 << 20)
        g2 = ix.search(c.w.queries, c.w.exclude_ids, 64, -1.0, 4, 32, with_stats=True)
        assert g2[3].pool_retries == 0 and g2[3].pool_entries == st.pool_entries
        for x, y in zip(g2[:3], (g_ids, g_sc, g_pr)):
            assert np.array_equal(x.cpu().numpy(), y)
    finally:
        ix.close()
    o = c.oracle(64, -1.0, 4, 32)
    rep = compare(g_ids, g_sc, g_pr, o)
    print(f"[gpu-test] low tau -> {rep}", flush=True)
    assert_parity(rep)


def test_invalid_arguments_leave_outputs_untouched():
    ps = _lib()
    c = case("tiny")
    q = c.w.queries
    for kw in (dict(k=0), dict(k=65), dict(W=0), dict(nprobe_max=0), dict(tau=float("nan"))):
        args = dict(k=10, tau=0.9, W=3, nprobe_max=12)
        args.update(kw)
        with pytest.raises(ps.SieveError) as e:
            c.ix.search(q, c.w.exclude_ids, args["k"], args["tau"], args["W"],
                        args["nprobe_max"])
        assert e.value.code == -1


@pytest.mark.parametrize("name", ["tiny", "tiny16", "c1"])
def test_rank_order_matches_oracle_exactly(name):
    """Kernel (1): the probe order equals the oracle's fp64 order, all ranks."""
    c = case(name)
    nl = c.w.spec.nlist
    P = c.ix.rank(c.w.queries, nl).cpu().numpy()
    h = c.h
    o = oracle.search(h["vectors"], h["list_offsets"], h["ids"], h["centroids"], h["queries"],
                      h["exclude_ids"], 1, 2.0, 1, nl, want_order=True, nthreads=NTHREADS)
    assert np.array_equal(P, o.order)


@pytest.mark.parametrize("name", ["tiny", "tiny16", "c1"])
def test_rank_prefix_matches_oracle_exactly(name, rank_path):
    """Short prefixes of the probe order (the lazily ranked part) equal the oracle's."""
    c = case(name)
    nl = c.w.spec.nlist
    h = c.h
    o = oracle.search(h["vectors"], h["list_offsets"], h["ids"], h["centroids"], h["queries"],
                      h["exclude_ids"], 1, 2.0, 1, nl, want_order=True, nthreads=NTHREADS)
    for R in sorted({1, 8, min(nl, 32), min(nl, 64)}):
        P = c.ix.rank(c.w.queries, R).cpu().numpy()
        assert np.array_equal(P, o.order[:, :R]), R


@pytest.mark.parametrize("name", ["tiny", "tiny16", "c1"])
@pytest.mark.parametrize("lookahead", [True, False])
def test_sieve_matches_oracle_on_each_rank_path(name, lookahead, rank_path):
    c = case(name)
    s = c.w.spec
    _check(c, s.k, s.tau, s.W, s.nprobe_max, lookahead)


@pytest.mark.parametrize("nlist,d,dtype", [(2048, 32, torch.float32), (5000, 64, torch.float16),
                                           (1500, 128, torch.float16)])
def test_rank_and_search_on_large_centroid_sets(nlist, d, dtype, rank_path):
    """More than 1,024 centroids: long prefixes take the register-resident block selector,
    short ones the fused screen (or the materialised path, forced); the order must be the
    oracle's exactly and a search with nprobe = 150 must match it."""
    rng = np.random.default_rng(nlist)
    n, nq = 30000, 96
    C = rng.standard_normal((nlist, d))
    C /= np.linalg.norm(C, axis=1, keepdims=True)
    X = rng.standard_normal((n, d))
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    npdt = np.float32 if dtype == torch.float32 else np.float16
    C, X = C.astype(npdt), X.astype(npdt)
    lab = rng.integers(0, nlist, n)
    order = np.argsort(lab, kind="stable")
    X = X[order]
    off = np.concatenate([[0], np.cumsum(np.bincount(lab, minlength=nlist))]).astype(np.int64)
    ids = order.astype(np.int64)
    qrows = rng.choice(n, nq, replace=False)
    Q = X[qrows].copy()
    ex = ids[qrows]
    ps = _lib()
    dev = "cuda"
    ix = ps.Index(torch.from_numpy(X).to(dev), torch.from_numpy(off).to(dev),
                  torch.from_numpy(ids).to(dev), torch.from_numpy(C).to(dev))
    try:
        tq = torch.from_numpy(Q).to(dev)
        o = oracle.search(X, off, ids, C, Q, ex, 1, 2.0, 1, 300, want_order=True,
                          nthreads=NTHREADS)
        for R in (8, 64, 100, 300):
            P = ix.rank(tq, R).cpu().numpy()
            assert np.array_equal(P, o.order[:, :R]), R
        g = ix.search(tq, torch.from_numpy(ex).to(dev), 10, 0.5, 4, 150)
        og = oracle.search(X, off, ids, C, Q, ex, 10, 0.5, 4, 150, nthreads=NTHREADS)
        assert_parity(compare(g[0].cpu().numpy(), g[1].cpu().numpy(), g[2].cpu().numpy(), og))
        f = ix.search_fixed(tq, torch.from_numpy(ex).to(dev), 10, 0.5, 150)
        of = oracle.search(X, off, ids, C, Q, ex, 10, 0.5, oracle.W_INF, 150, nthreads=NTHREADS)
        assert_parity(compare(f[0].cpu().numpy(), f[1].cpu().numpy(), f[2].cpu().numpy(), of))
    finally:
        ix.close()


@pytest.fixture(params=[1, 2, 4])
def pass1_div(request):
    """The register-query prefix bounds the R-th score from the first 1/div of the
    centroids (1: all of them); a looser bound admits more candidates, and a query whose
    candidates overflow its buffer is re-ranked by the wide fallback."""
    old = os.environ.get("SIEVE_RANK_PASS1_DIV")
    os.environ["SIEVE_RANK_PASS1_DIV"] = str(request.param)
    yield request.param
    if old is None:
        os.environ.pop("SIEVE_RANK_PASS1_DIV", None)
    else:
        os.environ["SIEVE_RANK_PASS1_DIV"] = old


@pytest.mark.parametrize("R", [8, 32, 33, 64])
def test_rank_prefix_on_many_work_groups(R, rank_path, pass1_div):
    """128-dim fp16 queries on a large centroid set: the fused prefix keeps the queries of
    each wave in registers, 128 queries per work-group; 1,100 queries span nine
    work-groups, the last one ragged (76 queries); R runs from 8 to the 64-rank maximum
    of the fused prefix.  The order is exact whatever part of the centroids bounds the
    first pass."""
    rng = np.random.default_rng(900 + R)
    nlist, d, nq = 1800, 128, 1100
    C = rng.standard_normal((nlist, d))
    C /= np.linalg.norm(C, axis=1, keepdims=True)
    Q = rng.standard_normal((nq, d))
    Q /= np.linalg.norm(Q, axis=1, keepdims=True)
    C, Q = C.astype(np.float16), Q.astype(np.float16)
    X = C[:4].copy()  # a token index: only the order is checked
    off = np.zeros(nlist + 1, np.int64)
    off[1:] = 4
    ids = np.arange(4, dtype=np.int64)
    ps = _lib()
    ix = ps.Index(torch.from_numpy(X).cuda(), torch.from_numpy(off).cuda(),
                  torch.from_numpy(ids).cuda(), torch.from_numpy(C).cuda())
    try:
        P = ix.rank(torch.from_numpy(Q).cuda(), R).cpu().numpy()
    finally:
        ix.close()
    o = oracle.search(X, off, ids, C, Q, None, 1, 2.0, 1, R, want_order=True, nthreads=NTHREADS)
    print(f"[gpu-test] rank prefix R={R} path={rank_path} pass-1 div={pass1_div}", flush=True)
    assert np.array_equal(P, o.order[:, :R])


def test_rank_with_many_exact_ties_takes_the_wide_path(rank_path):
    """800 identical centroids tie at the top: the one-wave selection runs out of
    boundary room, the search re-ranks with the wide kernel, and the order is
    still the oracle's (ties to the lower centroid index)."""
    rng = np.random.default_rng(11)
    d, nlist, n = 32, 1024, 3000
    C = rng.standard_normal((nlist, d)).astype(np.float32)
    C /= np.linalg.norm(C, axis=1, keepdims=True)
    C[100:900] = C[100]
    X = rng.standard_normal((n, d)).astype(np.float32)
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    sizes = rng.multinomial(n, np.ones(nlist) / nlist)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    ids = np.arange(n, dtype=np.int64)
    Q = (C[100] + 0.01 * rng.standard_normal((64, d))).astype(np.float32)
    Q /= np.linalg.norm(Q, axis=1, keepdims=True)
    ps = _lib()
    dev = "cuda"
    ix = ps.Index(torch.from_numpy(X).to(dev), torch.from_numpy(off).to(dev),
                  torch.from_numpy(ids).to(dev), torch.from_numpy(C).to(dev))
    P = ix.rank(torch.from_numpy(Q).to(dev), 16).cpu().numpy()
    o = oracle.search(X, off, ids, C, Q, None, 1, 2.0, 1, 16, want_order=True)
    assert np.array_equal(P, o.order)
    g = ix.search(torch.from_numpy(Q).to(dev), None, 10, 0.5, 3, 16)
    o = oracle.search(X, off, ids, C, Q, None, 10, 0.5, 3, 16)
    assert_parity(compare(g[0].cpu().numpy(), g[1].cpu().numpy(), g[2].cpu().numpy(), o))


def test_round_log_matches_stats():
    """sieve_round_log: one record per round whose sums are the search's statistics."""
    c = case("c1")
    s = c.w.spec
    for kw in (dict(lookahead=True), dict(lookahead=False), dict(lookahead=True,
                                                                  speculative=True)):
        r = c.ix.search(c.w.queries, c.w.exclude_ids, s.k, 0.5, s.W, s.nprobe_max,
                        with_stats=True, **kw)
        st = r[3]
        log = c.ix.round_log()
        assert len(log) == st.rounds
        assert sum(x.items for x in log) == st.items
        assert sum(x.item_rows for x in log) == st.vectors_scanned
        assert sum(x.list_loads for x in log) == st.list_loads
        assert sum(x.candidates for x in log) == st.hits
        assert all(x.ms_scan > 0 and x.kind == 0 for x in log)
        assert abs(sum(x.ms_scan for x in log) - st.ms_scan) <= 1e-3 * max(st.ms_scan, 1.0)
    f = c.ix.search_fixed(c.w.queries, c.w.exclude_ids, s.k, s.tau, s.nprobe_max,
                          with_stats=True)
    log = c.ix.round_log()
    assert len(log) == f[3].rounds and all(x.kind == 1 for x in log)
    assert sum(x.items for x in log) == f[3].items


def test_pool_index_limit_gives_a_clean_error():
    """A search that would hold more candidate-pool slots than the final merge can index
    fails with SIEVE_EUNSUPPORTED before the merge runs; the limit is lowered through its
    knob so that no large pool is needed, and the handle keeps working afterwards."""
    ps = _lib()
    c = case("c1")
    s = c.w.spec
    os.environ["SIEVE_POOL_LIMIT"] = "1000"
    try:
        with pytest.raises(ps.SieveError) as e:
            c.ix.search(c.w.queries, c.w.exclude_ids, s.k, 0.3, s.W, s.nprobe_max)
        assert e.value.code == -4 and "candidate-pool entries" in str(e.value)
    finally:
        del os.environ["SIEVE_POOL_LIMIT"]
    _check(c, s.k, s.tau, s.W, s.nprobe_max)


def test_workspace_cap_gives_enomem():
    """A workspace allocation the device cannot serve fails the call with SIEVE_ENOMEM and a
    message, before any launch that needs it; the allocation cap is forced through its knob
    (no real exhaustion).  The same handle then searches normally, with the result of an
    index that never failed."""
    ps = _lib()
    c = case("c1")
    s = c.w.spec
    q, ex = c.w.queries, c.w.exclude_ids
    ix = ps.Index(c.w.vectors, c.w.list_offsets, c.w.ids, c.w.centroids)
    try:
        # 16x the batch: the workspace the handle holds (sized at load) must grow
        qq, exx = q.repeat(16, 1).contiguous(), ex.repeat(16).contiguous()
        os.environ["SIEVE_ALLOC_CAP"] = "4096"
        try:
            for call in (lambda: ix.search(qq, exx, s.k, s.tau, s.W, s.nprobe_max),
                         lambda: ix.search_fixed(qq, exx, s.k, s.tau, s.fixed_nprobe)):
                with pytest.raises(ps.SieveError) as e:
                    call()
                assert e.value.code == -2 and "SIEVE_ALLOC_CAP" in str(e.value)
        finally:
            del os.environ["SIEVE_ALLOC_CAP"]
        got = [t.cpu().numpy() for t in ix.search(q, ex, s.k, s.tau, s.W, s.nprobe_max)]
        want = [t.cpu().numpy() for t in c.ix.search(q, ex, s.k, s.tau, s.W, s.nprobe_max)]
        for x, y in zip(got, want):
            assert np.array_equal(x, y)
    finally:
        ix.close()


@pytest.mark.parametrize("k", [1, 10, 64])
@pytest.mark.parametrize("fixed", [False, True])
@pytest.mark.parametrize("knob", [None, ("SIEVE_SPILL_CAP", "0"), ("SIEVE_ARENA", "0")])
def test_candidate_memory_bounded_by_k_per_tile(k, fixed, knob):
    """Local results keep at most k candidates per (query, tile): at tau = 0.1 about a third
    of the scanned rows qualify, yet the pool holds at most k entries per (query, row chunk).
    A tile's qualifying rows go to its work-group's candidate arena (LDS, then a global
    extension), and each query's exact top k is selected from it at the end of the tile.
    With the extension removed, tiles whose rows overflow the LDS arena, and with the arena
    off, all tiles with candidates, take the exact top-k pass instead.  The result equals
    the oracle's every way."""
    c = case("c1")
    s = c.w.spec
    q, ex = c.w.queries, c.w.exclude_ids
    ix = c.ix
    if knob is not None:
        # the knobs are read when a search sizes its workspace: a fresh index
        ps = _lib()
        os.environ[knob[0]] = knob[1]
        ix = ps.Index(c.w.vectors, c.w.list_offsets, c.w.ids, c.w.centroids)
    try:
        if fixed:
            r = ix.search_fixed(q, ex, k, 0.1, s.nprobe_max, with_stats=True)
        else:
            r = ix.search(q, ex, k, 0.1, s.W, s.nprobe_max, with_stats=True)
    finally:
        if knob is not None:
            del os.environ[knob[0]]
            ix.close()
    st = r[3]
    off = c.h["list_offsets"]
    chunks = int(np.ceil(np.diff(off).max() / 512))
    print(f"[gpu-test] k={k} fixed={fixed} knob={knob}: found {st.hits}, pool "
          f"{st.pool_entries}, heavy records {st.heavy_records}, items {st.items}", flush=True)
    assert st.pool_entries <= k * st.items * chunks
    assert st.hits > st.pool_entries
    if knob is not None:
        assert st.heavy_records > 0
    else:
        assert st.heavy_records == 0
    o = c.oracle(k, 0.1, oracle.W_INF if fixed else s.W, s.nprobe_max)
    rep = compare(r[0].cpu().numpy(), r[1].cpu().numpy(), r[2].cpu().numpy(), o)
    print(f"[gpu-test] -> {rep}", flush=True)
    assert_parity(rep)
