"""Seeded synthetic workloads for threshold-aware IVF search.

This module only *makes inputs*: a mixture-of-Gaussians corpus on the unit
sphere with planted near-duplicate groups, a spherical k-means IVF build with
exact nearest-centroid assignment (the build precondition of Sec. 4.4), and a
query sample drawn from the corpus (a self-join; each query's own row id is
passed as its exclusion id).  It holds none of the search method's
arithmetic: no probe order, no partition scan, no stop rule, no merge.  Both
the GPU path and the CPU oracle consume what it produces.

Everything is drawn from named, seeded sub-streams, so a (spec, seed, device)
triple always gives the same arrays.  Generation runs on the CPU or on a GPU
through PyTorch (large corpora need the GPU for k-means and assignment); the
two devices draw different random streams, so a dataset is only ever compared
against itself.

Recipe (the stand-in for the paper's corpora, Sec. 3.1 and Sec. 6.1):
  * centres c_m = normalize(N(0, I_d)), m = 0..n_comp-1; each row picks m
    uniformly and is x = normalize(c_m + sigma * z), z ~ N(0, I_d);
  * near-duplicate groups are carved from a random permutation of the rows
    until the grouped rows reach dup_frac * N (the last group is cut to at
    least 2); a group's first row is its seed and keeps its vector, every
    other member becomes normalize(seed + sigma_g * z);
  * vectors are then rounded to the storage dtype (fp32 or fp16);
  * spherical k-means: nlist distinct sample rows as the initial centroids,
    then `iters` rounds of (argmax inner-product assignment, mean,
    normalize); an empty cluster keeps its previous centroid; centroids are
    rounded to the storage dtype;
  * exact assignment of every row to its highest-inner-product stored
    centroid (fp32 screen, fp64 re-check of near-ties, lowest index wins);
  * rows are stored partition-major, sorted by (list, row id); ids are the
    original row indices;
  * queries: Q distinct rows, uniformly without replacement; exclude_ids are
    their row ids.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Optional

import numpy as np
import torch

__all__ = ["WorkloadSpec", "Workload", "SPECS", "make", "list_stats"]


@dataclasses.dataclass(frozen=True)
class WorkloadSpec:
    name: str
    n: int
    d: int
    dtype: str  # "f32" | "f16"
    n_comp: int
    sigma: float
    dup_frac: float
    dup_size: tuple  # ("uniform", lo, hi) | ("geom", p) | ("zipf", a, cap)
    dup_sigma: tuple  # (const,) | (lo, hi) drawn per group
    nlist: int
    kmeans_sample: int  # 0 = all rows
    kmeans_iters: int
    nq: int
    k: int
    tau: float
    W: int
    nprobe_max: int
    fixed_nprobe: int
    seed: int


SPECS = {
    # small cases for the CPU test suite
    "tiny": WorkloadSpec("tiny", 3000, 32, "f32", 30, 0.3, 0.15, ("uniform", 2, 8), (0.02,),
                         16, 0, 10, 150, 10, 0.90, 3, 12, 12, 7),
    "tiny16": WorkloadSpec("tiny16", 3000, 64, "f16", 30, 0.25, 0.15, ("uniform", 2, 8),
                           (0.02,), 16, 0, 10, 150, 10, 0.90, 3, 12, 12, 8),
    # tiny self-join, the oracle runs in seconds
    "c1": WorkloadSpec("c1", 20_000, 64, "f32", 200, 0.3, 0.10, ("uniform", 2, 8), (0.02,),
                       64, 0, 10, 1_000, 10, 0.90, 8, 32, 32, 1001),
    # mid-size self-join (also the data of the W / tau / nprobe sweep)
    "c2": WorkloadSpec("c2", 1_000_000, 128, "f32", 2_000, 0.25, 0.15, ("geom", 1.0 / 3.0),
                       (0.015,), 1_024, 100_000, 10, 10_000, 10, 0.92, 8, 128, 128, 1002),
    # 10M x 768 fp16 dedup-shaped workload
    "c3": WorkloadSpec("c3", 10_000_000, 768, "f16", 20_000, 0.2, 0.20, ("zipf", 1.5, 1000),
                       (0.01, 0.03), 4_096, 500_000, 10, 100_000, 10, 0.95, 8, 256, 256, 1003),
    # 100M x 128 fp16, 25.6 GB resident
    "c5": WorkloadSpec("c5", 100_000_000, 128, "f16", 100_000, 0.25, 0.10, ("zipf", 1.5, 500),
                       (0.02,), 16_384, 1_000_000, 10, 1_000_000, 10, 0.90, 8, 512, 512, 1005),
}


@dataclasses.dataclass
class Workload:
    spec: WorkloadSpec
    vectors: torch.Tensor  # [N, d] storage dtype, partition-major
    ids: torch.Tensor  # [N] int64
    list_offsets: torch.Tensor  # [nlist + 1] int64
    centroids: torch.Tensor  # [nlist, d] storage dtype
    queries: torch.Tensor  # [Q, d] storage dtype
    exclude_ids: torch.Tensor  # [Q] int64
    assign_refined: int = 0  # rows whose assignment needed the fp64 re-check

    def numpy(self) -> dict:
        """Host copies (fp16 stays fp16) for the CPU oracle."""
        return {k: getattr(self, k).cpu().numpy() for k in
                ("vectors", "ids", "list_offsets", "centroids", "queries", "exclude_ids")}

    def to(self, device) -> "Workload":
        return dataclasses.replace(self, **{k: getattr(self, k).to(device) for k in
                                            ("vectors", "ids", "list_offsets", "centroids",
                                             "queries", "exclude_ids")})


def _torch_dtype(s: str):
    return {"f32": torch.float32, "f16": torch.float16}[s]


def _gen(seed: int, stream: str, device) -> torch.Generator:
    h = hashlib.sha256(f"{seed}/{stream}".encode()).digest()
    g = torch.Generator(device=device)
    g.manual_seed(int.from_bytes(h[:8], "little") & ((1 << 63) - 1))
    return g


def _np_rng(seed: int, stream: str) -> np.random.Generator:
    h = hashlib.sha256(f"{seed}/{stream}".encode()).digest()
    return np.random.Generator(np.random.Philox(int.from_bytes(h[:8], "little")))


def _normalize(x: torch.Tensor) -> torch.Tensor:
    return x / x.norm(dim=1, keepdim=True).clamp_min(1e-30)


def _group_sizes(spec: WorkloadSpec, rng: np.random.Generator) -> np.ndarray:
    target = int(round(spec.dup_frac * spec.n))
    if target < 2:
        return np.zeros(0, np.int64)
    kind = spec.dup_size[0]
    out, total = [], 0
    while total < target:
        m = max(1024, (target - total) // 2)
        if kind == "uniform":
            s = rng.integers(spec.dup_size[1], spec.dup_size[2] + 1, size=m)
        elif kind == "geom":
            s = 1 + rng.geometric(spec.dup_size[1], size=m)
        elif kind == "zipf":
            s = np.minimum(1 + rng.zipf(spec.dup_size[1], size=m), spec.dup_size[2])
        else:
            raise ValueError(kind)
        out.append(s.astype(np.int64))
        total += int(s.sum())
    sizes = np.concatenate(out)
    cs = np.cumsum(sizes)
    last = int(np.searchsorted(cs, target))  # first group where the cumsum reaches target
    sizes = sizes[: last + 1].copy()
    before = int(cs[last - 1]) if last > 0 else 0
    sizes[-1] = max(2, target - before)
    return sizes


def _rows(n, chunk):
    for a in range(0, n, chunk):
        yield a, min(n, a + chunk)


@torch.no_grad()
def _argmax_ip(x_store: torch.Tensor, c_store: torch.Tensor, margin: float, chunk: int):
    """Exact highest-inner-product centroid per row, lowest index on ties."""
    n = x_store.shape[0]
    out = torch.empty(n, dtype=torch.int64, device=x_store.device)
    cf = c_store.float()
    refined = 0
    for a, b in _rows(n, chunk):
        xs = x_store[a:b].float()
        s = xs @ cf.T
        top = torch.topk(s, 2, dim=1) if cf.shape[0] > 1 else None
        if top is None:
            out[a:b] = 0
            continue
        best = top.indices[:, 0]
        near = (top.values[:, 0] - top.values[:, 1]) <= margin
        if bool(near.any()):
            rows = near.nonzero().flatten()
            s64 = xs[rows].double() @ c_store.double().T
            mx = s64.max(dim=1, keepdim=True).values
            # first index attaining the maximum
            cand = torch.where(s64 == mx, torch.arange(cf.shape[0], device=xs.device),
                               torch.full_like(s64, cf.shape[0], dtype=torch.int64))
            best[rows] = cand.min(dim=1).values
            refined += int(rows.numel())
        out[a:b] = best
    return out, refined


@torch.no_grad()
def make(spec: WorkloadSpec | str, device: Optional[str] = None, seed: Optional[int] = None,
         nq: Optional[int] = None) -> Workload:
    """Build the seeded workload described by ``spec`` on ``device``."""
    if isinstance(spec, str):
        spec = SPECS[spec]
    if seed is not None or nq is not None:
        spec = dataclasses.replace(spec, seed=spec.seed if seed is None else seed,
                                   nq=spec.nq if nq is None else nq)
    if device is None:
        device = "cuda" if torch.cuda.is_available() else "cpu"
    dev = torch.device(device)
    N, d, s = spec.n, spec.d, spec.seed
    sdt = _torch_dtype(spec.dtype)
    chunk = max(1, (1 << 26) // d)              # rows per elementwise chunk
    mchunk = max(1, (1 << 28) // spec.nlist)    # rows per (rows x nlist) score block

    # mixture corpus
    g_c = _gen(s, "centres", dev)
    centres = _normalize(torch.randn(spec.n_comp, d, generator=g_c, device=dev))
    g_m = _gen(s, "membership", dev)
    member = torch.randint(spec.n_comp, (N,), generator=g_m, device=dev)
    g_z = _gen(s, "noise", dev)
    x = torch.empty(N, d, dtype=torch.float32, device=dev)
    for a, b in _rows(N, chunk):
        x[a:b] = _normalize(centres[member[a:b]] +
                            spec.sigma * torch.randn(b - a, d, generator=g_z, device=dev))
    del member

    # near-duplicate groups
    rng = _np_rng(s, "dup-groups")
    sizes = _group_sizes(spec, rng)
    if sizes.size:
        g_p = _gen(s, "dup-rows", dev)
        perm = torch.randperm(N, generator=g_p, device=dev)
        starts = np.concatenate([[0], np.cumsum(sizes)[:-1]])
        if len(spec.dup_sigma) == 1:
            gsig = np.full(sizes.size, spec.dup_sigma[0])
        else:
            gsig = rng.uniform(spec.dup_sigma[0], spec.dup_sigma[1], size=sizes.size)
        # member m of group g (m >= 1) sits at perm[starts[g] + m]
        mem_group = np.repeat(np.arange(sizes.size), sizes - 1)
        mem_pos = (np.arange(int((sizes - 1).sum())) -
                   np.repeat(np.cumsum(sizes - 1) - (sizes - 1), sizes - 1) +
                   np.repeat(starts, sizes - 1) + 1)
        mem_rows = perm[torch.from_numpy(mem_pos).to(dev)]
        seed_rows = perm[torch.from_numpy(starts[mem_group]).to(dev)]
        sig = torch.from_numpy(gsig[mem_group]).to(dev, torch.float32)
        g_dz = _gen(s, "dup-noise", dev)
        for a, b in _rows(mem_rows.numel(), chunk):
            x[mem_rows[a:b]] = _normalize(x[seed_rows[a:b]] + sig[a:b, None] *
                                          torch.randn(b - a, d, generator=g_dz, device=dev))
        del perm, mem_rows, seed_rows, sig
    xs_store = x.to(sdt) if sdt != torch.float32 else x
    del x

    # spherical k-means on a sample
    g_k = _gen(s, "kmeans-sample", dev)
    ns = N if spec.kmeans_sample <= 0 else min(N, spec.kmeans_sample)
    samp = torch.randperm(N, generator=g_k, device=dev)[:ns]
    xsamp = xs_store[samp].float()
    cent = xsamp[: spec.nlist].clone()
    for _ in range(spec.kmeans_iters):
        assign = torch.empty(ns, dtype=torch.int64, device=dev)
        for a, b in _rows(ns, mchunk):
            assign[a:b] = (xsamp[a:b] @ cent.T).argmax(dim=1)
        sums, cnt = _cluster_sums(xsamp, assign, spec.nlist)
        keep = cnt == 0
        newc = _normalize(sums)
        cent = torch.where(keep[:, None], cent, newc)
    del xsamp, samp
    c_store = cent.to(sdt) if sdt != torch.float32 else cent

    # exact assignment, partition-major layout
    margin = 4.0 * d * 2.0 ** -24 + 1e-7
    assign, refined = _argmax_ip(xs_store, c_store, margin, mchunk)
    order = torch.sort(assign, stable=True).indices
    counts = torch.bincount(assign, minlength=spec.nlist)
    offsets = torch.zeros(spec.nlist + 1, dtype=torch.int64, device=dev)
    offsets[1:] = torch.cumsum(counts, 0)
    vectors = xs_store[order]
    ids = order.to(torch.int64)
    del assign

    # queries: distinct rows of the corpus, self excluded by id
    g_q = _gen(s, "queries", dev)
    qrows = torch.randperm(N, generator=g_q, device=dev)[: spec.nq]
    queries = xs_store[qrows].clone()
    del xs_store
    return Workload(spec, vectors.contiguous(), ids, offsets, c_store.contiguous(),
                    queries.contiguous(), qrows.to(torch.int64), refined)


def _cluster_sums(x: torch.Tensor, assign: torch.Tensor, k: int):
    """Per-cluster sums of the rows of x, in a fixed order (no float atomics, so the same
    inputs give the same bits in every process): rows sorted by cluster (stable), fp64
    prefix sums, differences at the cluster boundaries."""
    order = torch.sort(assign, stable=True).indices
    cnt = torch.bincount(assign, minlength=k)
    ends = torch.cumsum(cnt, 0)
    pre = torch.zeros(x.shape[0] + 1, x.shape[1], dtype=torch.float64, device=x.device)
    pre[1:] = torch.cumsum(x[order].double(), 0)
    sums = (pre[ends] - pre[ends - cnt]).float()
    return sums, cnt


def list_stats(list_offsets) -> dict:
    """Partition occupancy statistics (CV, Gini, max/mean) of an index (Table 1 analogue)."""
    sizes = np.diff(np.asarray(list_offsets, dtype=np.int64)).astype(np.float64)
    mean = sizes.mean()
    srt = np.sort(sizes)
    n = srt.size
    gini = (2.0 * np.sum((np.arange(1, n + 1)) * srt) / (n * srt.sum()) - (n + 1) / n) \
        if srt.sum() > 0 else 0.0
    return {"lists": int(n), "mean": float(mean), "cv": float(sizes.std() / mean) if mean else 0.0,
            "gini": float(gini), "max_over_mean": float(sizes.max() / mean) if mean else 0.0,
            "empty": int((sizes == 0).sum())}
