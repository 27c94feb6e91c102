"""GPU parity of the multi-index search (Sec. 6.1's coarse shards, each with its own IVF and
stop rule, one global top-k merge) against the oracle's merge of per-shard searches."""
import os

import numpy as np
import pytest
import torch

import oracle
import sieve_workloads as sw
from parity import assert_parity, compare

pytestmark = pytest.mark.gpu

NTHREADS = min(16, os.cpu_count() or 1)


def _shards(h, parts, seed):
    """Rows of one index split into independently built indexes (same centroids)."""
    rng = np.random.default_rng(seed)
    owner = rng.integers(0, parts, len(h["ids"]))
    off = np.asarray(h["list_offsets"])
    lists = np.repeat(np.arange(len(off) - 1), np.diff(off))
    out = []
    for p in range(parts):
        rows = np.nonzero(owner == p)[0]
        cnt = np.bincount(lists[rows], minlength=len(off) - 1)
        out.append({"vectors": np.ascontiguousarray(h["vectors"][rows]),
                    "ids": np.ascontiguousarray(h["ids"][rows]),
                    "list_offsets": np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64),
                    "centroids": np.ascontiguousarray(h["centroids"])})
    return out


@pytest.fixture(scope="module")
def sharded():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2608_03199_amd as ps
    ps.load_library()
    print("[gpu-test] generating workload c1 and 4 shards", flush=True)
    w = sw.make("c1", device="cuda")
    h = w.numpy()
    shards = _shards(h, 4, 17)
    ixs = [ps.Index(torch.from_numpy(s["vectors"]).cuda(), torch.from_numpy(s["list_offsets"]).cuda(),
                    torch.from_numpy(s["ids"]).cuda(), torch.from_numpy(s["centroids"]).cuda())
           for s in shards]
    yield w, h, shards, ixs
    for ix in ixs:
        ix.close()


@pytest.mark.parametrize("W,tau", [(8, 0.9), (2, 0.9), (4, 0.6), (oracle.W_INF, 0.9)])
def test_multi_index_matches_oracle(sharded, W, tau):
    import paper_2608_03199_amd as ps
    w, h, shards, ixs = sharded
    s = w.spec
    g = ps.search_multi(ixs, w.queries, w.exclude_ids, s.k, tau, W, s.nprobe_max,
                        with_stats=True)
    o = oracle.search_multi(shards, h["queries"], h["exclude_ids"], s.k, tau, W, s.nprobe_max,
                            nthreads=NTHREADS)
    rep = compare(g[0].cpu().numpy(), g[1].cpu().numpy(), g[2].cpu().numpy(), o)
    print(f"[gpu-test] multi W={W} tau={tau} -> {rep}", flush=True)
    assert_parity(rep)
    assert g[3].probes_total == int(g[2].sum())
    # the dispatch never changes results
    for kw in (dict(lookahead=False), dict(serial=True)):
        b = ps.search_multi(ixs, w.queries, w.exclude_ids, s.k, tau, W, s.nprobe_max, **kw)
        for x, y in zip(g[:3], b):
            assert torch.equal(x, y)


def test_multi_index_of_one_equals_plain_search(sharded):
    import paper_2608_03199_amd as ps
    w, h, shards, ixs = sharded
    s = w.spec
    a = ps.search_multi(ixs[:1], w.queries, w.exclude_ids, s.k, s.tau, s.W, s.nprobe_max)
    b = ixs[0].search(w.queries, w.exclude_ids, s.k, s.tau, s.W, s.nprobe_max)
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    with pytest.raises(ps.SieveError):
        ps.search_multi(ixs, w.queries, w.exclude_ids, 0, s.tau, s.W, s.nprobe_max)


@pytest.mark.parametrize("eps", [0.05, 0.005])
def test_multi_index_calibrated_per_shard(sharded, eps):
    """Per-shard calibration (Appendix A): every shard replays its own fixed-probe outcomes on
    the same sampled query indices and chooses its own W.  Each chosen W equals the oracle's
    replay of that shard's sample; the sampled queries carry the merge of the shards'
    fixed-probe results and the other queries the merge of each shard's search with its own
    W, both against the oracle."""
    import paper_2608_03199_amd as ps
    w, h, shards, ixs = sharded
    s = w.spec
    rng = np.random.default_rng(1234)
    smp = np.sort(rng.choice(s.nq, s.nq // 10, replace=False)).astype(np.int32)
    ids, sc, pr, Ws = ps.search_multi_calibrated(ixs, w.queries, w.exclude_ids, s.k, s.tau,
                                                 s.nprobe_max, torch.from_numpy(smp).cuda(), eps)
    ids, sc, pr = ids.cpu().numpy(), sc.cpu().numpy(), pr.cpu().numpy()
    qs, xs = h["queries"][smp], h["exclude_ids"][smp]
    want, edge = [], 0
    for sh in shards:
        o = oracle.search(sh["vectors"], sh["list_offsets"], sh["ids"], sh["centroids"], qs, xs,
                          s.k, s.tau, oracle.W_INF, s.nprobe_max, oracle.MODE_A, NTHREADS,
                          want_hitseq=True)
        wo, _, _ = oracle.calibrate(o.hitseq, o.rank, eps)
        want.append(8 if wo is None else wo)
        edge += int((o.flags & oracle.FLAG_TAU_EDGE).astype(bool).sum())
    print(f"[gpu-test] multi calibrated eps={eps}: W {Ws}, oracle {want}, tau-edge {edge}",
          flush=True)
    if edge == 0:
        assert Ws == want
    of = oracle.search_multi(shards, qs, xs, s.k, s.tau, oracle.W_INF, s.nprobe_max,
                             nthreads=NTHREADS)
    rep = compare(ids[smp], sc[smp], pr[smp], of)
    print(f"[gpu-test] multi calibrated sample -> {rep}", flush=True)
    assert_parity(rep)
    rest = np.setdiff1d(np.arange(s.nq), smp)
    orr = oracle.search_multi(shards, h["queries"][rest], h["exclude_ids"][rest], s.k, s.tau,
                              list(Ws), s.nprobe_max, nthreads=NTHREADS)
    rep = compare(ids[rest], sc[rest], pr[rest], orr)
    print(f"[gpu-test] multi calibrated rest -> {rep}", flush=True)
    assert_parity(rep)
