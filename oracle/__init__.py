"""Test infrastructure only: ctypes binding to the plain C fp64 oracle.

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg import this package.  The GPU library never imports,
links or calls it, and the two share no code.

``build()`` compiles ``sieve_oracle.c`` with gcc into ``liboracle.so`` next to
it (flags below: no fast-math, no FP contraction).  Arrays are numpy arrays
on the host; fp16 data are passed as raw ``uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sieve_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
CFLAGS = ["-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math"]

F32, F16 = 0, 1
MODE_A, MODE_B = 0, 1
W_INF = 0x7FFFFFFF
FLAG_TAU_EDGE, FLAG_KTH_TIE, FLAG_ORDER_TIE, FLAG_CENTROID_TIE = 1, 2, 4, 8

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (always recompiles when ``force``)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm", "-lpthread"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        # SIEVE_ORACLE_LIB: another build of the same source (the sanitizer test)
        path = os.environ.get("SIEVE_ORACLE_LIB", _LIB)
        if path == _LIB and not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        lib.oracle_search.restype = ctypes.c_int
        lib.oracle_search.argtypes = [P, ctypes.c_int, i64, ctypes.c_int, P, ctypes.c_int, P, P,
                                      P, i64, P, ctypes.c_int, ctypes.c_float, ctypes.c_int,
                                      ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      P, P, P, P, P, P, P, P, P, P]
        lib.oracle_bruteforce.restype = ctypes.c_int
        lib.oracle_bruteforce.argtypes = [P, ctypes.c_int, i64, ctypes.c_int, P, P, i64, P,
                                          ctypes.c_int, ctypes.c_float, ctypes.c_int, P, P, P]
        lib.oracle_calibrate.restype = ctypes.c_int
        lib.oracle_calibrate.argtypes = [i64, ctypes.c_int, ctypes.c_int, P, P, ctypes.c_double,
                                         P, P]
        lib.oracle_half_to_double.restype = ctypes.c_double
        lib.oracle_half_to_double.argtypes = [ctypes.c_uint16]
        del i32
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype in (np.float16, np.uint16):
        return F16
    raise TypeError(f"unsupported dtype {a.dtype}")


def _raw(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a)
    return a.view(np.uint16) if a.dtype == np.float16 else a


class OracleResult(dict):
    __getattr__ = dict.__getitem__


def search(vectors, list_offsets, ids, centroids, queries, exclude_ids, k, tau, W, nprobe_max,
           mode=MODE_A, nthreads=1, want_hitseq=False, want_order=False) -> OracleResult:
    """Threshold-aware IVF search, sequential per query (modes A and B)."""
    lib = _load()
    vectors = _raw(vectors)
    centroids = _raw(centroids)
    queries = _raw(queries)
    dt = _dtype_code(vectors)
    n_vec, d = vectors.shape
    nlist = centroids.shape[0]
    nq = queries.shape[0]
    list_offsets = np.ascontiguousarray(list_offsets, dtype=np.int64)
    ids = np.ascontiguousarray(ids, dtype=np.int64)
    ex = None if exclude_ids is None else np.ascontiguousarray(exclude_ids, dtype=np.int64)
    n = min(int(nprobe_max), nlist)
    r = OracleResult(
        ids=np.empty((nq, k), np.int64), scores=np.empty((nq, k), np.float64),
        probes=np.empty(nq, np.int32), flags=np.empty(nq, np.int32),
        last_hit=np.empty(nq, np.int32), scanned=np.empty(nq, np.int64),
        ncand=np.empty(nq, np.int64), rank=np.empty((nq, k), np.int32),
        hitseq=np.empty((nq, n), np.uint8) if want_hitseq else None,
        order=np.empty((nq, n), np.int32) if want_order else None)
    st = lib.oracle_search(_ptr(vectors), dt, n_vec, d, _ptr(list_offsets), nlist, _ptr(ids),
                           _ptr(centroids), _ptr(queries), nq, _ptr(ex), int(k),
                           ctypes.c_float(tau), int(W), int(nprobe_max), int(mode), int(nthreads),
                           _ptr(r.ids), _ptr(r.scores), _ptr(r.probes), _ptr(r.flags),
                           _ptr(r.last_hit), _ptr(r.hitseq), _ptr(r.order), _ptr(r.scanned),
                           _ptr(r.ncand), _ptr(r.rank))
    if st != 0:
        raise RuntimeError(f"oracle_search failed with status {st}")
    return r


def search_fixed(vectors, list_offsets, ids, centroids, queries, exclude_ids, k, tau, nprobe,
                 nthreads=1, **kw) -> OracleResult:
    """Fixed-probe baseline: the same traversal with no stop rule."""
    return search(vectors, list_offsets, ids, centroids, queries, exclude_ids, k, tau, W_INF,
                  nprobe, MODE_A, nthreads, **kw)


def bruteforce(vectors, ids, queries, exclude_ids, k, tau, nthreads=1) -> OracleResult:
    """Exhaustive filtered top-k over every row (no IVF)."""
    lib = _load()
    vectors = _raw(vectors)
    queries = _raw(queries)
    dt = _dtype_code(vectors)
    n_vec, d = vectors.shape
    nq = queries.shape[0]
    ids = np.ascontiguousarray(ids, dtype=np.int64)
    ex = None if exclude_ids is None else np.ascontiguousarray(exclude_ids, dtype=np.int64)
    r = OracleResult(ids=np.empty((nq, k), np.int64), scores=np.empty((nq, k), np.float64),
                     count=np.empty(nq, np.int64))
    st = lib.oracle_bruteforce(_ptr(vectors), dt, n_vec, d, _ptr(ids), _ptr(queries), nq, _ptr(ex),
                               int(k), ctypes.c_float(tau), int(nthreads), _ptr(r.ids),
                               _ptr(r.scores), _ptr(r.count))
    if st != 0:
        raise RuntimeError(f"oracle_bruteforce failed with status {st}")
    return r


def search_multi(shards, queries, exclude_ids, k, tau, W, nprobe_max, mode=MODE_A, nthreads=1):
    """Search over several independently built indexes (Sec. 6.1's coarse shards): each shard
    runs the threshold search with its own stop rule (oracle.search), and the per-query union
    of the shard results is ordered by (score desc, id asc) and cut to k.  shards: a list of
    dicts with vectors, list_offsets, ids, centroids.  probes = the sum over the shards.
    The tie flags are recomputed on the merged list; TAU_EDGE and KTH_TIE of any shard are
    kept (a shard's (k+1)-th candidate never reaches the merge).  W: one window for every
    shard, or a list with one per shard (per-shard calibration, Appendix A)."""
    Ws = list(W) if isinstance(W, (list, tuple)) else [W] * len(shards)
    parts = [search(sh["vectors"], sh["list_offsets"], sh["ids"], sh["centroids"], queries,
                    exclude_ids, k, tau, w, nprobe_max, mode, nthreads)
             for sh, w in zip(shards, Ws)]
    nq = np.asarray(queries).shape[0]
    r = OracleResult(ids=np.full((nq, k), -1, np.int64), scores=np.full((nq, k), -np.inf),
                     probes=np.zeros(nq, np.int32), flags=np.zeros(nq, np.int32))
    for i in range(nq):
        cand = [(float(p.scores[i, j]), int(p.ids[i, j])) for p in parts for j in range(k)
                if p.ids[i, j] >= 0]
        cand.sort(key=lambda t: (-t[0], t[1]))
        for j, (sc, cid) in enumerate(cand[:k]):
            r.ids[i, j] = cid
            r.scores[i, j] = sc
        r.probes[i] = sum(int(p.probes[i]) for p in parts)
        f = 0
        for p in parts:
            f |= int(p.flags[i]) & (FLAG_TAU_EDGE | FLAG_KTH_TIE)
        if len(cand) > k and cand[k - 1][0] - cand[k][0] < 1e-4:
            f |= FLAG_KTH_TIE
        if any(cand[j][0] - cand[j + 1][0] < 1e-4 for j in range(min(k, len(cand)) - 1)):
            f |= FLAG_ORDER_TIE
        r.flags[i] = f
    return r


def calibrate(hitseq, found_rank, eps):
    """Required-window histogram and chosen W from recorded fixed-probe outcomes."""
    lib = _load()
    hitseq = np.ascontiguousarray(hitseq, dtype=np.uint8)
    found_rank = np.ascontiguousarray(found_rank, dtype=np.int32)
    ns, n = hitseq.shape
    k = found_rank.shape[1]
    hist = np.zeros(n + 1, np.int64)
    z = np.zeros(1, np.int64)
    w = lib.oracle_calibrate(ns, n, k, _ptr(hitseq), _ptr(found_rank), float(eps), _ptr(hist),
                             _ptr(z))
    if w == -1:
        raise RuntimeError("oracle_calibrate: bad arguments")
    return (None if w == -2 else int(w)), hist, int(z[0])


def half_to_double(bits: int) -> float:
    return float(_load().oracle_half_to_double(int(bits)))
