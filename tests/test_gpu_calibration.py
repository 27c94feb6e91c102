"""GPU parity of the in-call window calibration (Appendix A, Algorithm 3).

The library samples nothing itself: the test draws the sample (seeded,
uniform without replacement) and passes it in.  The oracle then does the
whole procedure on the CPU, independently of the HIP path: a fixed-probe
search of the sampled queries recording each probe's outcome, the replay of
the stop rule over those outcomes (oracle.calibrate), and a threshold search
of every other query with the chosen window.  Checked: the chosen window
equals the oracle's (for several loss targets, which pins the histogram's
prefix sums); the sampled queries' outputs equal the oracle's fixed-probe
ones, the other queries' equal the oracle's search with that window (ids and
probes exact, scores within 1e-4, tests/parity.py).
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


@pytest.fixture(scope="module", autouse=True)
def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2608_03199_amd as ps
    ps.load_library()


_cases = {}


def _case(name):
    if name not in _cases:
        import paper_2608_03199_amd as ps
        print(f"[gpu-test] generating workload {name}", flush=True)
        w = sw.make(name, device="cuda")
        _cases[name] = (w, w.numpy(), ps.Index(w.vectors, w.list_offsets, w.ids, w.centroids))
    return _cases[name]


def _oracle_search(h, sel, k, tau, W, nprobe, want_hitseq=False):
    ex = None if h["exclude_ids"] is None else h["exclude_ids"][sel]
    return oracle.search(h["vectors"], h["list_offsets"], h["ids"], h["centroids"],
                         h["queries"][sel], ex, k, tau, W, nprobe, oracle.MODE_A, NTHREADS,
                         want_hitseq=want_hitseq)


def _sample(nq, ns, seed):
    rng = np.random.default_rng(seed)
    return rng.choice(nq, ns, replace=False).astype(np.int32)


def _run_and_check(name, ns, eps, tau=None, fallback=8, seed=0):
    w, h, ix = _case(name)
    s = w.spec
    tau = s.tau if tau is None else tau
    nq = s.nq
    smp = _sample(nq, ns, seed)
    eps32 = float(np.float32(eps))
    ids, sc, pr, W = (x.cpu().numpy() if torch.is_tensor(x) else x for x in
                      ix.search_calibrated(w.queries, w.exclude_ids, s.k, tau, s.nprobe_max,
                                           torch.from_numpy(smp).cuda(), eps32, fallback))
    # oracle: fixed-probe sample with recorded outcomes, replay, choose
    of = _oracle_search(h, smp, s.k, tau, oracle.W_INF, s.nprobe_max, want_hitseq=True)
    w_or, hist, z = oracle.calibrate(of.hitseq, of.rank, eps32) if ns else (None, None, 0)
    want_W = fallback if w_or is None else w_or
    tau_edge = int((of.flags & oracle.FLAG_TAU_EDGE).astype(bool).sum()) if ns else 0
    print(f"[gpu-test] calibrated {name} ns={ns} eps={eps} tau={tau}: W gpu={W} oracle={want_W} "
          f"z={z} tau_edge_in_sample={tau_edge}", flush=True)
    if tau_edge == 0:
        assert W == want_W
    if ns:
        rep = compare(ids[smp], sc[smp], pr[smp], of)
        print(f"[gpu-test]   sample -> {rep}", flush=True)
        assert_parity(rep)
    rest = np.setdiff1d(np.arange(nq), smp)
    if rest.size:
        orest = _oracle_search(h, rest, s.k, tau, W, s.nprobe_max)
        rep = compare(ids[rest], sc[rest], pr[rest], orest)
        print(f"[gpu-test]   rest (W={W}) -> {rep}", flush=True)
        assert_parity(rep)
    return ids, sc, pr, W


# Thresholds: the workloads' own (near-duplicates, found mostly at rank 1)
# and lower ones whose neighbours spread over many ranks, so that the
# required windows cover a range of values.
@pytest.mark.parametrize("name,tau", [("tiny", 0.9), ("tiny", 0.6), ("tiny16", 0.5),
                                      ("c1", 0.9), ("c1", 0.5)])
@pytest.mark.parametrize("eps", [0.3, 0.05, 0.005])
def test_calibrated_search_matches_oracle(name, tau, eps):
    nq = sw.SPECS[name].nq
    _run_and_check(name, ns=max(30, nq // 10), eps=eps, tau=tau, seed=11)


def test_calibrated_window_tracks_loss_target():
    # a finer sweep of targets on one workload: each chooses the oracle's W,
    # and the chosen windows differ (the histogram's prefix sums are pinned)
    ws = [_run_and_check("c1", ns=200, eps=eps, tau=0.5, seed=3)[3]
          for eps in (0.5, 0.2, 0.1, 0.05, 0.02, 0.01, 0.005, 0.001)]
    print(f"[gpu-test] windows by target: {ws}", flush=True)
    assert ws == sorted(ws) and len(set(ws)) >= 3


def test_calibration_edges():
    import paper_2608_03199_amd as ps
    w, h, ix = _case("tiny")
    s = w.spec
    nq = s.nq
    # empty sample: the fallback window over the whole batch, equal to a plain search
    ids, sc, pr, W = ix.search_calibrated(w.queries, w.exclude_ids, s.k, s.tau, s.nprobe_max,
                                          torch.empty(0, dtype=torch.int32, device="cuda"),
                                          0.01, 5)
    assert W == 5
    b = ix.search(w.queries, w.exclude_ids, s.k, s.tau, 5, s.nprobe_max)
    for x, y in zip((ids, sc, pr), b):
        assert torch.equal(x, y)
    # every query sampled: the fixed-probe result, and the oracle's window
    ids, sc, pr, W = _run_and_check("tiny", ns=nq, eps=0.01, seed=5)
    f = ix.search_fixed(w.queries, w.exclude_ids, s.k, s.tau, s.nprobe_max)
    for x, y in zip((ids, sc, pr), f):
        assert np.array_equal(x, y.cpu().numpy())
    # no neighbour anywhere (tau above every score): the fallback window
    _, _, pr, W = _run_and_check("tiny", ns=20, eps=0.01, tau=1.5, fallback=3, seed=6)
    assert W == 3
    # a single sampled query, ragged
    _run_and_check("tiny16", ns=1, eps=0.2, seed=9)
    # invalid samples are rejected
    bad = [np.array([0, 0], np.int32), np.array([-1], np.int32), np.array([nq], np.int32)]
    for smp in bad:
        with pytest.raises(ps.SieveError) as e:
            ix.search_calibrated(w.queries, w.exclude_ids, s.k, s.tau, s.nprobe_max,
                                 torch.from_numpy(smp).cuda(), 0.01, 8)
        assert e.value.code == -1
    for eps in (0.0, -0.1, 1.5, float("nan")):
        with pytest.raises(ps.SieveError):
            ix.search_calibrated(w.queries, w.exclude_ids, s.k, s.tau, s.nprobe_max,
                                 torch.arange(4, dtype=torch.int32, device="cuda"), eps, 8)


def test_calibrated_search_is_repeatable():
    w, h, ix = _case("c1")
    s = w.spec
    smp = torch.from_numpy(_sample(s.nq, 40, 21)).cuda()
    a = ix.search_calibrated(w.queries, w.exclude_ids, s.k, s.tau, s.nprobe_max, smp, 0.01)
    b = ix.search_calibrated(w.queries, w.exclude_ids, s.k, s.tau, s.nprobe_max, smp, 0.01)
    assert a[3] == b[3]
    for x, y in zip(a[:3], b[:3]):
        assert torch.equal(x, y)
