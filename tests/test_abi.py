"""CPU-side checks of the C ABI: the library builds for gfx950, loads, exports
every symbol include/sieve.h declares, mirrors sieve_stats exactly, and
rejects bad arguments before any HIP call."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sieve.h")


@pytest.fixture(scope="module")
def lib():
    import paper_2608_03199_amd as ps
    if not os.path.exists(ps.LIB_PATH):
        from paper_2608_03199_amd import build
        build.build()
    return ps.load_library()


def declared_symbols():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"SIEVE_API\s+[\w\s\*]+?\b(sieve_\w+)\s*\(", txt)))


def test_header_declares_the_boundary():
    syms = declared_symbols()
    for s in ("sieve_load_index", "sieve_search", "sieve_search_fixed", "sieve_search_calibrated",
              "sieve_search_multi", "sieve_round_log", "sieve_free_index", "sieve_last_error"):
        assert s in syms


def test_library_exports_every_declared_symbol(lib):
    import paper_2608_03199_amd as ps
    out = subprocess.run(["nm", "-D", "--defined-only", ps.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (sieve_\w+)", out))
    assert set(declared_symbols()) <= exported
    for s in declared_symbols():
        assert hasattr(lib, s)
    # nothing else with C linkage leaks out
    assert all(s.startswith("sieve_") for s in exported)


def test_stats_struct_layout_matches_c(tmp_path):
    import paper_2608_03199_amd as ps
    fields = [f for f, _ in ps.Stats._fields_]
    src = tmp_path / "layout.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "sieve.h"\nint main(void){'
                   'printf("%zu", sizeof(sieve_stats));' +
                   "".join(f'printf(" %zu", offsetof(sieve_stats, {f}));' for f in fields) +
                   "return 0;}\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    vals = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(ps.Stats)
    assert vals[1:] == [getattr(ps.Stats, f).offset for f in fields]


def test_round_struct_layout_matches_c(tmp_path):
    import paper_2608_03199_amd as ps
    fields = [f for f, _ in ps.Round._fields_]
    src = tmp_path / "round.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "sieve.h"\nint main(void){'
                   'printf("%zu", sizeof(sieve_round));' +
                   "".join(f'printf(" %zu", offsetof(sieve_round, {f}));' for f in fields) +
                   "return 0;}\n")
    exe = tmp_path / "round"
    subprocess.run(["gcc", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    vals = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(ps.Round)
    assert vals[1:] == [getattr(ps.Round, f).offset for f in fields]


def test_argument_errors_without_a_gpu(lib):
    # no handle: rejected before any HIP call
    rc = lib.sieve_search(None, None, 0, None, 10, 0.9, 8, 32, 1, None, None, None, None, None)
    assert rc == -1 and b"NULL" in lib.sieve_last_error()
    rc = lib.sieve_search_fixed(None, None, 0, None, 10, 0.9, 32, None, None, None, None, None)
    assert rc == -1
    w = ctypes.c_int32(-7)
    rc = lib.sieve_search_calibrated(None, None, 0, None, 10, 0.9, 32, None, 0, 0.005, 8, None,
                                     None, None, ctypes.byref(w), None, None)
    assert rc == -1 and w.value == -7
    rc = lib.sieve_search_multi(None, 0, None, 0, None, 10, 0.9, 8, 32, 1, None, None, None,
                                None, None)
    assert rc == -1
    n = ctypes.c_int32(-3)
    rc = lib.sieve_round_log(None, None, 0, ctypes.byref(n))
    assert rc == -1 and n.value == -3
    h = ctypes.c_void_p()
    rc = lib.sieve_load_index(None, 0, 10, 64, None, 4, None, None, None, ctypes.byref(h))
    assert rc == -1 and h.value is None
    rc = lib.sieve_load_index(None, 7, 0, 64, None, 4, None, None, None, ctypes.byref(h))
    assert rc == -1 and b"dtype" in lib.sieve_last_error()
    fake = ctypes.c_void_p(0x1000)
    rc = lib.sieve_load_index(fake, 0, 0, 12, fake, 4, fake, fake, None, ctypes.byref(h))
    assert rc == -4  # d not a multiple of 8
    rc = lib.sieve_load_index(fake, 0, 0, 64, fake, 20000, fake, fake, None, ctypes.byref(h))
    assert rc == -4  # nlist above the supported maximum
    lib.sieve_free_index(None)
    assert b"gfx950" in lib.sieve_version()


def test_no_cpu_fallback_in_binding():
    """The binding holds marshalling only: no oracle import, no torch compute on the path."""
    src = open(os.path.join(ROOT, "paper_2608_03199_amd", "__init__.py")).read()
    assert "oracle" not in src.replace("no oracle", "")
    for bad in ("torch.topk", "torch.matmul", "@", "torch.sort", ".mm("):
        assert bad not in src.split('"""', 2)[2]


def test_pool_index_limit_host_rule(tmp_path):
    """The candidate-pool guard: a search may hold at most 2^38 pool slots (a sanity bound
    far above device memory: the final merge uses 64-bit offsets); the override only lowers
    the limit."""
    src = tmp_path / "limits.cpp"
    src.write_text(
        '#include <stdio.h>\n#include "host_limits.h"\nusing namespace sieve;\nint main(){'
        'printf("%lld %lld %lld %lld %lld\\n", (long long)pool_index_limit(0),'
        ' (long long)pool_index_limit(""), (long long)pool_index_limit("1000"),'
        ' (long long)pool_index_limit("-5"), (long long)pool_index_limit("99999999999"));'
        'printf("%d %d %d %d\\n", pool_slots_fit(274877906944ull, pool_index_limit(0)),'
        ' pool_slots_fit(274877906945ull, pool_index_limit(0)), pool_slots_fit(1000, 1000),'
        ' pool_slots_fit(1001, 1000));return 0;}\n')
    exe = tmp_path / "limits"
    csrc = os.path.join(ROOT, "paper_2608_03199_amd", "csrc")
    subprocess.run(["g++", "-std=c++17", "-Wall", "-Werror", "-I", csrc, str(src), "-o",
                    str(exe)], check=True)
    lines = subprocess.run([str(exe)], capture_output=True, text=True,
                           check=True).stdout.split("\n")
    assert lines[0].split() == ["274877906944", "274877906944", "1000", "274877906944",
                                "99999999999"]
    assert lines[1].split() == ["1", "0", "1", "0"]
