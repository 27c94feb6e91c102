"""The allocation-free ranking entry point (sieve_rank_noalloc) against sieve_rank.

Both are called through the C ABI on the same seeded inputs; the probe orders must be
identical, element by element (integer output).  Two calls in a row share the library's
fixed device scratch: the second, with fewer queries, must not see the first's leftovers.
Both ranking paths are covered: the fused prefix path (nlist > 1024, short prefixes) and the
materialised screen path (forced through SIEVE_RANK_PATH=1).
"""
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ps():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2608_03199_amd as ps
    ps.load_library()
    return ps


def _index(ps, n, d, nlist, dtype, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    x = torch.randn((n, d), generator=g)
    x = (x / x.norm(dim=1, keepdim=True)).to(dtype).cuda()
    c = torch.randn((nlist, d), generator=g)
    c = (c / c.norm(dim=1, keepdim=True)).to(dtype).cuda()
    off = (torch.arange(nlist + 1, dtype=torch.int64) * (n // nlist)).cuda()
    off[-1] = n
    ids = torch.arange(n, dtype=torch.int64).cuda()
    return ps.Index(x, off, ids, c), g


def _queries(g, nq, d, dtype):
    q = torch.randn((nq, d), generator=g)
    return (q / q.norm(dim=1, keepdim=True)).to(dtype).cuda().contiguous()


@pytest.mark.parametrize("path", ["prefix", "screen"])
@pytest.mark.parametrize("dtype", [torch.float16, torch.float32])
def test_rank_noalloc_matches_rank(ps, path, dtype):
    old = os.environ.get("SIEVE_RANK_PATH")
    if path == "screen":
        os.environ["SIEVE_RANK_PATH"] = "1"
    try:
        ix, g = _index(ps, 60000, 128, 2048, dtype, seed=71)
        try:
            for nq, nprobe in ((5000, 48), (1234, 20)):
                q = _queries(g, nq, 128, dtype)
                want = ix.rank(q, nprobe)
                out = torch.full((nq, min(nprobe, ix.nlist)), -7, dtype=torch.int32,
                                 device=q.device)
                got = ix.rank_noalloc(q, nprobe, out)
                torch.cuda.synchronize()
                print(f"[gpu-test] rank_noalloc {path} {dtype} nq={nq} nprobe={nprobe}", flush=True)
                assert torch.equal(got.cpu(), want.cpu())
        finally:
            ix.close()
    finally:
        if old is None:
            os.environ.pop("SIEVE_RANK_PATH", None)
        else:
            os.environ["SIEVE_RANK_PATH"] = old


def test_rank_noalloc_argument_errors(ps):
    ix, g = _index(ps, 4000, 64, 32, torch.float32, seed=5)
    try:
        q = _queries(g, 10, 64, torch.float32)
        lib = ps.load_library()
        # a NULL output with queries: a clean error, nothing launched
        rc = lib.sieve_rank_noalloc(ix._h, q.data_ptr(), 10, 4, None, None)
        assert rc == -1
        assert b"non-NULL" in lib.sieve_last_error()
        # nq = 0 is a no-op
        assert lib.sieve_rank_noalloc(ix._h, None, 0, 4, None, None) == 0
    finally:
        ix.close()
