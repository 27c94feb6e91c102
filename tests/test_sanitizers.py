"""CPU sanitizer builds of the host-side C and C++ code.

* The oracle (oracle/sieve_oracle.c) is rebuilt with AddressSanitizer and
  UndefinedBehaviorSanitizer (any report aborts) and driven through its usual binding in a
  child process: threshold search in both modes and several threads, fixed probing,
  brute force, multi-index search, calibration, on fp32 and fp16 data with empty lists, W =
  infinity and nprobe > nlist.  The child's outputs must equal the normal build's.
* The host limit rules of the library (csrc/host_limits.h) run under the same sanitizers.
"""
import hashlib
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
       "-fno-omit-frame-pointer", "-g"]

# Runs in the child (and in this process with the normal build): prints one digest line.
DRIVER = r'''
import hashlib, sys
import numpy as np
sys.path.insert(0, ROOT)
import oracle

def digest(h, *arrs):
    for a in arrs:
        h.update(np.ascontiguousarray(a).tobytes())

rng = np.random.default_rng(11)
h = hashlib.sha256()
for dt in (np.float32, np.float16):
    n, d, nlist, nq = 900, 24, 12, 40
    x = rng.standard_normal((n, d)).astype(np.float32)
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    x[100:110] = x[5] + 0.01 * rng.standard_normal((10, d)).astype(np.float32)
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    c = x[rng.choice(n, nlist, replace=False)].copy()
    assign = np.argmax(x @ c.T, axis=1)
    assign[assign == 3] = 4  # list 3 empty
    order = np.argsort(assign, kind="stable")
    x = x[order].astype(dt)
    off = np.concatenate([[0], np.cumsum(np.bincount(assign, minlength=nlist))]).astype(np.int64)
    ids = (order * 7 + 3).astype(np.int64)
    qi = rng.choice(n, nq, replace=False)
    q = x[qi].copy()
    ex = ids[qi].copy()
    c = c.astype(dt)
    for mode in (oracle.MODE_A, oracle.MODE_B):
        for W, npm in ((2, 8), (oracle.W_INF, 20)):
            r = oracle.search(x, off, ids, c, q, ex, 5, 0.5, W, npm, mode, 3, want_hitseq=True)
            digest(h, r.ids, r.scores, r.probes, r.flags)
    f = oracle.search_fixed(x, off, ids, c, q, ex, 5, 0.5, 6)
    digest(h, f.ids, f.scores, f.probes)
    b = oracle.bruteforce(x, ids, q, ex, 7, 0.2, 2)
    digest(h, b.ids, b.scores)
    half = off[nlist // 2]
    shards = [dict(vectors=x[:half], list_offsets=off[:nlist // 2 + 1], ids=ids[:half],
                   centroids=c[:nlist // 2]),
              dict(vectors=x[half:], list_offsets=off[nlist // 2:] - half, ids=ids[half:],
                   centroids=c[nlist // 2:])]
    m = oracle.search_multi(shards, q, ex, 5, 0.5, 3, 6)
    digest(h, m.ids, m.scores, m.probes)
    r = oracle.search(x, off, ids, c, q, ex, 5, 0.5, oracle.W_INF, nlist, oracle.MODE_A, 1,
                      want_hitseq=True)
    w, _, z = oracle.calibrate(r.hitseq, r.rank, 0.05)
    h.update(repr((w, z)).encode())
print("DIGEST", h.hexdigest())
'''


def _run_driver(env):
    code = "ROOT = %r\n" % ROOT + DRIVER
    out = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                         timeout=300)
    assert out.returncode == 0, out.stderr[-4000:]
    return [l for l in out.stdout.splitlines() if l.startswith("DIGEST")][-1]


def _runtime(name):
    p = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True,
                       text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


def test_oracle_under_asan_ubsan(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("gcc sanitizer runtimes not installed")
    import oracle
    lib = tmp_path / "liboracle_san.so"
    subprocess.run(["gcc", *oracle.CFLAGS, *SAN, "-o", str(lib),
                    os.path.join(ROOT, "oracle", "sieve_oracle.c"), "-lm", "-lpthread"],
                   check=True)
    env = dict(os.environ)
    want = _run_driver(env)  # the normal build
    env.update(SIEVE_ORACLE_LIB=str(lib), LD_PRELOAD=f"{asan}:{ubsan}",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    got = _run_driver(env)
    assert got == want


def test_host_limits_under_asan_ubsan(tmp_path):
    if not _runtime("libasan.so"):
        pytest.skip("gcc sanitizer runtimes not installed")
    src = tmp_path / "limits.cpp"
    src.write_text(
        '#include <stdio.h>\n#include "host_limits.h"\nusing namespace sieve;\nint main(){'
        'const char* k[] = {nullptr, "", "0", "1", "1000", "-5", "abc", "99999999999",'
        ' "2147483647", "2147483648"};\n'
        'unsigned long long s[] = {0ull, 1ull, 1000ull, 2147483647ull, 2147483648ull,'
        ' ~0ull};\nlong long acc = 0;\n'
        'for (auto x : k) for (auto y : s) acc += pool_slots_fit(y, pool_index_limit(x));\n'
        'printf("%lld\\n", acc);return 0;}\n')
    exe = tmp_path / "limits"
    csrc = os.path.join(ROOT, "paper_2608_03199_amd", "csrc")
    subprocess.run(["g++", "-std=c++17", "-Wall", "-Werror", *SAN, "-I", csrc, str(src), "-o",
                    str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True,
                         env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0"))
    assert out.returncode == 0, out.stderr[-2000:]
    assert int(out.stdout.split()[0]) > 0
