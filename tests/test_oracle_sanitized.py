"""The oracle and the brute force built with AddressSanitizer and
UndefinedBehaviorSanitizer (host code only, gcc), run over small shapes that
reach every path: users sharing their parameters at both precisions, more
than 64 users, one CPU level, the longest chain, every search mode,
heterogeneous users, the outer grouping (both kinds of users), the stage-1
tables, single candidates, a grouping replay and the exhaustive search.

The sanitized library is loaded into a child Python process with the
sanitizer runtimes preloaded (the interpreter itself is not instrumented);
any invalid access or undefined operation aborts the child, and the test
fails with its report."""

import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import ctypes, sys
import numpy as np
sys.path.insert(0, __ROOT__)
import oracle
from paper_2504_14611_amd import workloads as W
lib = ctypes.CDLL(__SO__)
oracle._declare(lib)
oracle._lib = lib

def gen(name, n, **kw):
    w = W.WORKLOADS[name]
    if kw:
        w = w.replace(name="san", stream=950 + len(kw), num_instances=n, **kw)
    return W.generate(w, 0, n)

cases = [
    ("c0", gen("c0", 16)), ("c1", gen("c1", 16)), ("c1_f64", gen("c1", 8, dtype="f64")),
    ("c3", gen("c3", 4)), ("N70", gen("c4b", 2, N=70, L=8, K=8, J=8)),
    ("N129_f64", gen("c4b", 1, N=129, L=4, K=4, J=4, dtype="f64")),
    ("K1", gen("c1", 8, K=1, local_f=(2.0e9, 2.0e9))), ("J1", gen("c1", 8, J=1)),
    ("L255", gen("c1", 2, L=255, N=4, K=4, J=4, cycles=("lu", 1e5, 2e6))),
    ("p4a", gen("p4a", 8)), ("h1", gen("h1", 4)), ("h2", gen("h2", 4)),
]
for label, p in cases:
    for mode in (0, 1, 2, 4, 8, 9, 15):
        q = dict(p)
        q["mode"] = mode
        oracle.solve(q)
    if p.get("user_zeta") is None:
        t = oracle.user_tables(p)
    for inst in range(min(2, len(p["rate"]))):
        for s in (0, p["L"] - 1, p["L"]):
            oracle.eval_candidate(p, inst, s, p["J"] - 1, 1)
            oracle.eval_candidate(p, inst, s, 0, p["N"])
    print("ok", label, flush=True)

for label, p in (("g10", gen("g10", 3)), ("p5", gen("p5", 3)), ("h5", gen("h5", 2)),
                 ("g_N20", gen("g10", 1, N=20))):
    for mode in (0, 1, 8):
        q = dict(p)
        q["mode"] = mode
        g = oracle.solve_grouped(q)
        for inst in range(len(p["rate"])):
            G = int(g["num_groups"][inst])
            if G:
                oracle.eval_grouping(q, inst, g["group_end"][inst, :G], g["group_cut"][inst, :G],
                                     g["group_gpu_level"][inst, :G], g["group_batch"][inst, :G])
    print("ok", label, flush=True)

p = gen("c0", 4, N=4, L=3, K=3, J=2)
for inst in range(4):
    for suffix in (False, True):
        oracle.brute(p, inst, suffix_only=suffix)
ph = gen("h1", 2, N=4, L=3, K=3, J=2, dtype="f64")
for inst in range(2):
    oracle.brute(ph, inst, suffix_only=True)
print("ok brute", flush=True)
print("SANITIZED RUN COMPLETE", flush=True)
"""


def _runtime(name):
    path = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True,
                          text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.parametrize("front", [None, 2])
def test_oracle_and_brute_force_under_asan_and_ubsan(tmp_path, front):
    """front = 2: the grouping's fronts built with room for two states, so
    that their capacity rule runs on the p5 and h5 groupings."""
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not (asan and ubsan):
        pytest.skip("gcc sanitizer runtimes not installed")
    extra = [f"-DJO_FRONT={front}"] if front else []
    so = oracle.build(["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                       "-fno-omit-frame-pointer", "-g", *extra],
                      out=str(tmp_path / "libjdob_oracle_san.so"))
    env = dict(os.environ, LD_PRELOAD=f"{asan}:{ubsan}",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    code = CHILD.replace("__ROOT__", repr(ROOT)).replace("__SO__", repr(so))
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=600)
    assert r.returncode == 0 and "SANITIZED RUN COMPLETE" in r.stdout, \
        f"exit {r.returncode}\n{r.stdout[-2000:]}\n{r.stderr[-6000:]}"


def test_sanitizers_catch_a_planted_overrun(tmp_path):
    """The same run over a copy of the oracle that reads one element past
    the batch deadlines (lo[N+1]) must fail: the instrumentation is live."""
    import shutil
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not (asan and ubsan):
        pytest.skip("gcc sanitizer runtimes not installed")
    src = os.path.dirname(oracle.__file__)
    for f in oracle._SOURCES + oracle._HEADERS:
        shutil.copy(os.path.join(src, f), tmp_path / f)
    body = (tmp_path / "jdob_oracle_body.h").read_text()
    old = "REAL H = w->lo[b] - Phi;"
    assert body.count(old) == 1
    (tmp_path / "jdob_oracle_body.h").write_text(body.replace(old, "REAL H = w->lo[b + 1] - Phi;"))
    so = str(tmp_path / "lib_planted.so")
    subprocess.run(["gcc", *oracle.CFLAGS, "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-g", "-o", so, str(tmp_path / "jdob_oracle.c"), str(tmp_path / "jdob_brute.c"),
                    "-lm"], check=True)
    env = dict(os.environ, LD_PRELOAD=f"{asan}:{ubsan}",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1")
    code = CHILD.replace("__ROOT__", repr(ROOT)).replace("__SO__", repr(so))
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=600)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr
