"""Python binding of libsieve (threshold-aware IVF search on MI355X / gfx950).

Argument marshalling only: every step of a search runs in the HIP kernels of
``libsieve.so``.  Tensors are PyTorch CUDA (HIP) tensors; their device
pointers and torch's current stream are handed to the C ABI declared in
``include/sieve.h``.  There is no CPU fallback: importing works anywhere,
but constructing an index needs the built library and a GPU, and fails
loudly otherwise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

__all__ = ["SieveError", "Index", "Stats", "Round", "load_library", "LIB_PATH", "W_INF",
           "K_MAX", "F32", "F16", "search_multi", "LOOKAHEAD_OFF", "LOOKAHEAD_COMMITTED",
           "LOOKAHEAD_SERIAL", "LOOKAHEAD_SPECULATIVE"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsieve.so")
W_INF = 0x7FFFFFFF
K_MAX = 64
F32, F16 = 0, 1
# values of the lookahead argument (SIEVE_LOOKAHEAD_* in include/sieve.h)
LOOKAHEAD_OFF, LOOKAHEAD_COMMITTED, LOOKAHEAD_SERIAL, LOOKAHEAD_SPECULATIVE = 0, 1, 2, 3
_STATUS = {0: "SIEVE_OK", -1: "SIEVE_EINVAL", -2: "SIEVE_ENOMEM", -3: "SIEVE_EDEVICE",
           -4: "SIEVE_EUNSUPPORTED", -5: "SIEVE_EINTERNAL"}


class SieveError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_STATUS.get(code, code)}: {msg}")
        self.code = code


class Stats(ctypes.Structure):
    """Mirror of ``sieve_stats``."""
    _fields_ = [("rounds", ctypes.c_int32), ("nprobe_eff", ctypes.c_int32),
                ("scan_launches", ctypes.c_int32), ("pool_retries", ctypes.c_int32),
                ("items", ctypes.c_int64), ("probes_total", ctypes.c_int64),
                ("vectors_scanned", ctypes.c_int64), ("list_loads", ctypes.c_int64),
                ("hits", ctypes.c_int64), ("scan_bytes", ctypes.c_double),
                ("scan_flops", ctypes.c_double), ("rank_flops", ctypes.c_double),
                ("ms_rank", ctypes.c_float), ("ms_sched", ctypes.c_float),
                ("ms_scan", ctypes.c_float), ("ms_update", ctypes.c_float),
                ("ms_finalize", ctypes.c_float), ("ms_total", ctypes.c_float),
                ("pool_entries", ctypes.c_int64), ("heavy_records", ctypes.c_int64)]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


class Round(ctypes.Structure):
    """Mirror of ``sieve_round`` (one record of ``sieve_round_log``)."""
    _fields_ = [("items", ctypes.c_int64), ("list_rows", ctypes.c_int64),
                ("item_rows", ctypes.c_int64), ("list_loads", ctypes.c_int64),
                ("candidates", ctypes.c_int64), ("scan_bytes", ctypes.c_double),
                ("scan_flops", ctypes.c_double), ("ms_scan", ctypes.c_float),
                ("kind", ctypes.c_int32)]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


def _lookahead_code(lookahead: bool, speculative: bool, serial: bool) -> int:
    if serial:
        return LOOKAHEAD_SERIAL
    if not lookahead:
        return LOOKAHEAD_OFF
    return LOOKAHEAD_SPECULATIVE if speculative else LOOKAHEAD_COMMITTED


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libsieve.so (built by ``paper_2608_03199_amd.build``); raises if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise SieveError(-3, f"{path} is not built; run paper_2608_03199_amd/build.py "
                             "(there is no CPU fallback)")
    lib = ctypes.CDLL(path)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.sieve_load_index.restype = ctypes.c_int
    lib.sieve_load_index.argtypes = [P, i32, i64, i32, P, i32, P, P, P,
                                     ctypes.POINTER(ctypes.c_void_p)]
    lib.sieve_search.restype = ctypes.c_int
    lib.sieve_search.argtypes = [P, P, i64, P, i32, ctypes.c_float, i32, i32, i32, P, P, P,
                                 ctypes.POINTER(Stats), P]
    lib.sieve_search_fixed.restype = ctypes.c_int
    lib.sieve_search_fixed.argtypes = [P, P, i64, P, i32, ctypes.c_float, i32, P, P, P,
                                       ctypes.POINTER(Stats), P]
    lib.sieve_search_calibrated.restype = ctypes.c_int
    lib.sieve_search_calibrated.argtypes = [P, P, i64, P, i32, ctypes.c_float, i32, P, i64,
                                            ctypes.c_float, i32, P, P, P,
                                            ctypes.POINTER(ctypes.c_int32),
                                            ctypes.POINTER(Stats), P]
    lib.sieve_search_multi.restype = ctypes.c_int
    lib.sieve_search_multi.argtypes = [P, i32, P, i64, P, i32, ctypes.c_float, i32, i32, i32, P,
                                       P, P, ctypes.POINTER(Stats), P]
    lib.sieve_search_multi_calibrated.restype = ctypes.c_int
    lib.sieve_search_multi_calibrated.argtypes = [P, i32, P, i64, P, i32, ctypes.c_float, i32, P,
                                                  i64, ctypes.c_float, i32, P, P, P,
                                                  ctypes.POINTER(ctypes.c_int32),
                                                  ctypes.POINTER(Stats), P]
    lib.sieve_round_log.restype = ctypes.c_int
    lib.sieve_round_log.argtypes = [P, ctypes.POINTER(Round), i32, ctypes.POINTER(ctypes.c_int32)]
    lib.sieve_rank.restype = ctypes.c_int
    lib.sieve_rank.argtypes = [P, P, i64, i32, P, P]
    lib.sieve_rank_noalloc.restype = ctypes.c_int
    lib.sieve_rank_noalloc.argtypes = [P, P, i64, i32, P, P]
    lib.sieve_free_index.restype = None
    lib.sieve_free_index.argtypes = [P]
    lib.sieve_last_error.restype = ctypes.c_char_p
    lib.sieve_last_error.argtypes = []
    lib.sieve_version.restype = ctypes.c_char_p
    lib.sieve_version.argtypes = []
    _lib = lib
    return lib


def _check(lib, code: int):
    if code != 0:
        raise SieveError(code, lib.sieve_last_error().decode())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.float16:
        return F16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or float16)")


def _dev(t: torch.Tensor, name: str) -> torch.Tensor:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    return t.contiguous()


def _stream(stream) -> Optional[int]:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


class Index:
    """An IVF index copied into the library's device layout (``sieve_load_index``)."""

    def __init__(self, vectors: torch.Tensor, list_offsets: torch.Tensor, ids: torch.Tensor,
                 centroids: torch.Tensor, stream=None):
        lib = load_library()
        vectors = _dev(vectors, "vectors")
        centroids = _dev(centroids, "centroids")
        list_offsets = _dev(list_offsets.to(torch.int64), "list_offsets")
        ids = _dev(ids.to(torch.int64), "ids")
        if vectors.dim() != 2 or centroids.dim() != 2 or centroids.shape[1] != vectors.shape[1]:
            raise ValueError("vectors [n, d] and centroids [nlist, d] expected")
        if centroids.dtype != vectors.dtype:
            raise TypeError("vectors and centroids must share a dtype")
        self.dtype = vectors.dtype
        self.d = int(vectors.shape[1])
        self.n = int(vectors.shape[0])
        self.nlist = int(centroids.shape[0])
        self.device = vectors.device
        h = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check(lib, lib.sieve_load_index(vectors.data_ptr(), _dtype_code(vectors), self.n,
                                             self.d, list_offsets.data_ptr(), self.nlist,
                                             ids.data_ptr(), centroids.data_ptr(),
                                             _stream(stream), ctypes.byref(h)))
        self._h = h
        self._lib = lib

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.sieve_free_index(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _prep(self, queries, exclude_ids, k):
        queries = _dev(queries, "queries")
        if queries.dtype != self.dtype or queries.dim() != 2 or queries.shape[1] != self.d:
            raise ValueError(f"queries must be [nq, {self.d}] of {self.dtype}")
        nq = int(queries.shape[0])
        ex = None
        if exclude_ids is not None:
            ex = _dev(exclude_ids.to(torch.int64), "exclude_ids")
            if ex.numel() != nq:
                raise ValueError("exclude_ids must have one id per query")
        dev = queries.device
        out_ids = torch.empty((nq, max(int(k), 1)), dtype=torch.int64, device=dev)
        out_scores = torch.empty((nq, max(int(k), 1)), dtype=torch.float32, device=dev)
        out_probes = torch.empty((nq,), dtype=torch.int32, device=dev)
        return queries, ex, nq, out_ids, out_scores, out_probes

    def rank(self, queries: torch.Tensor, nprobe: int, stream=None) -> torch.Tensor:
        """Probe order: [nq, min(nprobe, nlist)] int32 centroid indices."""
        queries, _, nq, _, _, _ = self._prep(queries, None, 1)
        n = min(int(nprobe), self.nlist)
        out = torch.empty((nq, max(n, 1)), dtype=torch.int32, device=queries.device)
        with torch.cuda.device(self.device):
            _check(self._lib, self._lib.sieve_rank(self._h, queries.data_ptr(), nq, int(nprobe),
                                                   out.data_ptr(), _stream(stream)))
        return out[:, :n]

    def rank_noalloc(self, queries: torch.Tensor, nprobe: int, out: torch.Tensor,
                     stream=None) -> torch.Tensor:
        """``sieve_rank_noalloc`` into a caller-provided ``out`` ([nq, min(nprobe, nlist)]
        int32, contiguous, on the index's device); ``queries`` must already be contiguous in
        the index's dtype.  Neither this wrapper nor the library allocates."""
        n = min(int(nprobe), self.nlist)
        nq = int(queries.shape[0])
        if queries.dtype != self.dtype or not queries.is_contiguous() or queries.dim() != 2:
            raise SieveError(-1, "queries must be a contiguous [nq, d] tensor of the index dtype")
        if (out.dtype != torch.int32 or not out.is_contiguous()
                or tuple(out.shape) != (nq, n) or out.device != queries.device):
            raise SieveError(-1, f"out must be a contiguous int32 [{nq}, {n}] tensor on "
                                 "the queries' device")
        with torch.cuda.device(self.device):
            _check(self._lib, self._lib.sieve_rank_noalloc(self._h, queries.data_ptr(), nq,
                                                           int(nprobe), out.data_ptr(),
                                                           _stream(stream)))
        return out

    def round_log(self) -> list:
        """Per-round records (``Round``) of the last search on this index that collected
        statistics (``sieve_round_log``)."""
        n = ctypes.c_int32(0)
        _check(self._lib, self._lib.sieve_round_log(self._h, None, 0, ctypes.byref(n)))
        buf = (Round * max(n.value, 1))()
        _check(self._lib, self._lib.sieve_round_log(self._h, buf, n.value, ctypes.byref(n)))
        return [buf[i] for i in range(min(n.value, len(buf)))]

    def search(self, queries: torch.Tensor, exclude_ids: Optional[torch.Tensor], k: int,
               tau: float, W: int, nprobe_max: int, lookahead: bool = True,
               with_stats: bool = False, stream=None, serial: bool = False,
               speculative: bool = False):
        """Threshold-aware search; returns (ids, scores, probes[, Stats]).  lookahead:
        Algorithm 2 (else Algorithm 1); speculative: Algorithm 2 with speculative issue past
        the stop line; serial: the serial-traversal ablation (no shared partition scans;
        lookahead is ignored).  The outputs are the same in every mode."""
        queries, ex, nq, oi, osc, op = self._prep(queries, exclude_ids, k)
        st = Stats() if with_stats else None
        with torch.cuda.device(self.device):
            _check(self._lib, self._lib.sieve_search(
                self._h, queries.data_ptr(), nq, None if ex is None else ex.data_ptr(), int(k),
                float(tau), int(W), int(nprobe_max),
                _lookahead_code(lookahead, speculative, serial), oi.data_ptr(),
                osc.data_ptr(), op.data_ptr(), ctypes.byref(st) if st is not None else None,
                _stream(stream)))
        return (oi, osc, op, st) if with_stats else (oi, osc, op)

    def search_calibrated(self, queries: torch.Tensor, exclude_ids: Optional[torch.Tensor],
                          k: int, tau: float, nprobe_max: int, sample: torch.Tensor,
                          eps: float, W_fallback: int = 8, with_stats: bool = False,
                          stream=None):
        """Search whose window is chosen in the call from a fully probed sample
        (Appendix A, Algorithm 3).  sample: distinct int32 query indices on the
        queries' device.  Returns (ids, scores, probes, W[, Stats])."""
        queries, ex, nq, oi, osc, op = self._prep(queries, exclude_ids, k)
        smp = _dev(sample.to(torch.int32), "sample").reshape(-1)
        if smp.device != queries.device:
            raise ValueError("sample must be on the queries' device")
        st = Stats() if with_stats else None
        w = ctypes.c_int32(0)
        with torch.cuda.device(self.device):
            _check(self._lib, self._lib.sieve_search_calibrated(
                self._h, queries.data_ptr(), nq, None if ex is None else ex.data_ptr(), int(k),
                float(tau), int(nprobe_max), smp.data_ptr() if smp.numel() else None,
                int(smp.numel()), float(eps), int(W_fallback), oi.data_ptr(), osc.data_ptr(),
                op.data_ptr(), ctypes.byref(w), ctypes.byref(st) if st is not None else None,
                _stream(stream)))
        out = (oi, osc, op, int(w.value))
        return out + (st,) if with_stats else out

    def search_fixed(self, queries: torch.Tensor, exclude_ids: Optional[torch.Tensor], k: int,
                     tau: float, nprobe: int, with_stats: bool = False, stream=None):
        """Fixed-probe baseline; returns (ids, scores, probes[, Stats])."""
        queries, ex, nq, oi, osc, op = self._prep(queries, exclude_ids, k)
        st = Stats() if with_stats else None
        with torch.cuda.device(self.device):
            _check(self._lib, self._lib.sieve_search_fixed(
                self._h, queries.data_ptr(), nq, None if ex is None else ex.data_ptr(), int(k),
                float(tau), int(nprobe), oi.data_ptr(), osc.data_ptr(), op.data_ptr(),
                ctypes.byref(st) if st is not None else None, _stream(stream)))
        return (oi, osc, op, st) if with_stats else (oi, osc, op)


def search_multi(indexes, queries: torch.Tensor, exclude_ids: Optional[torch.Tensor], k: int,
                 tau: float, W: int, nprobe_max: int, lookahead: bool = True,
                 serial: bool = False, with_stats: bool = False, stream=None,
                 speculative: bool = False):
    """Threshold search over several independently built indexes of one corpus, each with its
    own stop rule, merged into one top-k (``sieve_search_multi``).  Returns
    (ids, scores, probes[, Stats]); probes are summed over the indexes."""
    indexes = list(indexes)
    if not indexes:
        raise ValueError("at least one index is required")
    first = indexes[0]
    queries, ex, nq, oi, osc, op = first._prep(queries, exclude_ids, k)
    handles = (ctypes.c_void_p * len(indexes))(*[ix._h.value for ix in indexes])
    st = Stats() if with_stats else None
    with torch.cuda.device(first.device):
        _check(first._lib, first._lib.sieve_search_multi(
            handles, len(indexes), queries.data_ptr(), nq, None if ex is None else ex.data_ptr(),
            int(k), float(tau), int(W), int(nprobe_max),
            _lookahead_code(lookahead, speculative, serial), oi.data_ptr(), osc.data_ptr(),
            op.data_ptr(), ctypes.byref(st) if st is not None else None, _stream(stream)))
    return (oi, osc, op, st) if with_stats else (oi, osc, op)


def search_multi_calibrated(indexes, queries: torch.Tensor, exclude_ids: Optional[torch.Tensor],
                            k: int, tau: float, nprobe_max: int, sample: torch.Tensor,
                            eps: float, W_fallback: int = 8, with_stats: bool = False,
                            stream=None):
    """``search_multi`` with the in-call window calibration (Appendix A) done per index on the
    same sampled query indices (``sieve_search_multi_calibrated``).  Returns
    (ids, scores, probes, [W per index][, Stats])."""
    indexes = list(indexes)
    if not indexes:
        raise ValueError("at least one index is required")
    first = indexes[0]
    queries, ex, nq, oi, osc, op = first._prep(queries, exclude_ids, k)
    smp = _dev(sample.to(torch.int32), "sample").reshape(-1)
    if smp.device != queries.device:
        raise ValueError("sample must be on the queries' device")
    handles = (ctypes.c_void_p * len(indexes))(*[ix._h.value for ix in indexes])
    ws = (ctypes.c_int32 * len(indexes))()
    st = Stats() if with_stats else None
    with torch.cuda.device(first.device):
        _check(first._lib, first._lib.sieve_search_multi_calibrated(
            handles, len(indexes), queries.data_ptr(), nq, None if ex is None else ex.data_ptr(),
            int(k), float(tau), int(nprobe_max), smp.data_ptr() if smp.numel() else None,
            int(smp.numel()), float(eps), int(W_fallback), oi.data_ptr(), osc.data_ptr(),
            op.data_ptr(), ws, ctypes.byref(st) if st is not None else None, _stream(stream)))
    out = (oi, osc, op, [int(x) for x in ws])
    return out + (st,) if with_stats else out
