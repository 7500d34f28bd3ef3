"""CPU oracle for batched J-DOB — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (``libjdob.so`` and
its binding) never calls it.

The oracle is plain C (``jdob_oracle.c``, ``jdob_oracle_body.h``) compiled
with gcc and ``-ffp-contract=off``; ``jdob_brute.c`` is an independent
exhaustive search used to pin it.  This module compiles them into
``libjdob_oracle.so`` next to the sources and wraps them with ctypes.  It
consumes the dicts produced by ``paper_2504_14611_amd.workloads.generate``
(numpy arrays) and shares no code with the GPU path.
"""

from __future__ import annotations

import ctypes as C
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libjdob_oracle.so")
_SOURCES = ["jdob_oracle.c", "jdob_brute.c"]
_HEADERS = ["jdob_oracle.h", "jdob_oracle_body.h", "jdob_oracle_hetero.h"]
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
          "-fno-fast-math", "-Wall", "-Wextra", "-Wno-unused-parameter"]


def build(extra_flags=(), out: str = _SO) -> str:
    """Compile the oracle with gcc into `out` (by default the library this
    module loads); returns its path."""
    srcs = [os.path.join(_HERE, s) for s in _SOURCES]
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", *CFLAGS, *extra_flags, "-o", tmp, *srcs, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def _stale() -> bool:
    if not os.path.exists(_SO):
        return True
    t = os.path.getmtime(_SO)
    return any(os.path.getmtime(os.path.join(_HERE, f)) > t for f in _SOURCES + _HEADERS)


_lib = None


def lib():
    global _lib
    if _lib is None:
        if _stale():
            build()
        _lib = C.CDLL(_SO)
        _declare(_lib)
    return _lib


def _problem_struct(real):
    P = C.POINTER(real)
    return type("jo_problem", (C.Structure,), {"_fields_": [
        ("I", C.c_int32), ("N", C.c_int32), ("L", C.c_int32), ("K", C.c_int32), ("J", C.c_int32),
        ("cycles", P), ("bits", P), ("alpha", P), ("beta", P), ("rate", P),
        ("deadline", P), ("t_free", P), ("local_freq", P), ("gpu_freq", P),
        ("kappa", C.c_double), ("p_tx", C.c_double), ("gpu_c", C.c_double),
        ("gpu_p_static", C.c_double), ("mode", C.c_int32),
        ("user_zeta", P), ("user_kappa", P), ("user_p_tx", P), ("user_local_freq", P)]})


# per-user parameters of heterogeneous users (optional keys of a problem dict)
USER_KEYS = ("user_zeta", "user_kappa", "user_p_tx", "user_local_freq")


def _policy_struct(real):
    P = C.POINTER(real)
    I32, I8, I64 = C.POINTER(C.c_int32), C.POINTER(C.c_int8), C.POINTER(C.c_int64)
    return type("jo_policy", (C.Structure,), {"_fields_": [
        ("status", I32), ("cut", I32), ("gpu_level", I32), ("batch", I32),
        ("energy", P), ("t_free_out", P), ("user_level", I8), ("user_offload", I8),
        ("energy_second", P), ("num_feasible", I32), ("num_user_evals", I64), ("user_freq", P)]})


def _tables_struct(real):
    P = C.POINTER(real)
    return type("jo_tables", (C.Structure,), {"_fields_": [
        ("order", C.POINTER(C.c_int16)), ("batch_deadline", P), ("min_batch", C.POINTER(C.c_int32)),
        ("uplink_time", P), ("gamma", P), ("self_level", C.POINTER(C.c_int8)),
        ("self_energy", P), ("self_slack", P)]})


def _grouped_struct(real):
    P = C.POINTER(real)
    I32, I16, I8, I64 = C.POINTER(C.c_int32), C.POINTER(C.c_int16), C.POINTER(C.c_int8), C.POINTER(C.c_int64)
    return type("jo_grouped", (C.Structure,), {"_fields_": [
        ("status", I32), ("num_groups", I32), ("energy", P), ("t_free_out", P),
        ("order", I16), ("group_end", I16), ("group_cut", I32), ("group_gpu_level", I32),
        ("group_batch", I32), ("group_energy", P), ("group_t_free", P),
        ("user_level", I8), ("user_offload", I8), ("user_group", I8),
        ("num_inner", I64), ("num_feasible", I64), ("num_user_evals", I64), ("user_freq", P)]})


def _grouping_struct(real):
    return type("jo_grouping", (C.Structure,), {"_fields_": [
        ("num_groups", C.c_int32), ("group_end", C.POINTER(C.c_int16)),
        ("group_cut", C.POINTER(C.c_int32)), ("group_gpu_level", C.POINTER(C.c_int32)),
        ("group_batch", C.POINTER(C.c_int32)), ("feasible", C.c_int32), ("energy", real),
        ("t_free_out", real), ("user_level", C.POINTER(C.c_int8)),
        ("user_offload", C.POINTER(C.c_int8)), ("user_freq", C.POINTER(real))]})


def _candidate_struct(real):
    return type("jo_candidate", (C.Structure,), {"_fields_": [
        ("feasible", C.c_int32), ("energy", real), ("t_free_out", real), ("gpu_latency", real),
        ("user_level", C.POINTER(C.c_int8)), ("user_offload", C.POINTER(C.c_int8)),
        ("user_freq", C.POINTER(real))]})


class _Brute(C.Structure):
    _fields_ = [("found", C.c_int32), ("energy", C.c_double), ("energy_second", C.c_double),
                ("cut", C.c_int32), ("gpu_level", C.c_int32), ("batch", C.c_int32),
                ("num_feasible", C.c_int32),
                ("user_level", C.POINTER(C.c_int8)), ("user_offload", C.POINTER(C.c_int8))]


_T = {}
for _sfx, _real in (("f32", C.c_float), ("f64", C.c_double)):
    _T[_sfx] = dict(real=_real, np=np.float32 if _sfx == "f32" else np.float64,
                    problem=_problem_struct(_real), policy=_policy_struct(_real),
                    tables=_tables_struct(_real), candidate=_candidate_struct(_real),
                    grouped=_grouped_struct(_real), grouping=_grouping_struct(_real))


def _declare(l):
    for sfx, t in _T.items():
        for name, argt in (("jo_solve", [C.POINTER(t["problem"]), C.c_int64, C.c_int64, C.POINTER(t["policy"])]),
                           ("jo_user_tables", [C.POINTER(t["problem"]), C.c_int64, C.c_int64, C.POINTER(t["tables"])]),
                           ("jo_eval_candidate", [C.POINTER(t["problem"]), C.c_int64, C.c_int, C.c_int, C.c_int,
                                                  C.POINTER(t["candidate"])]),
                           ("jo_solve_grouped", [C.POINTER(t["problem"]), C.c_int64, C.c_int64,
                                                 C.POINTER(t["grouped"])]),
                           ("jo_eval_grouping", [C.POINTER(t["problem"]), C.c_int64, C.POINTER(t["grouping"])])):
            fn = getattr(l, f"{name}_{sfx}")
            fn.argtypes = argt
            fn.restype = C.c_int
    l.jo_brute_f64.argtypes = [C.POINTER(_T["f64"]["problem"]), C.c_int64, C.c_int, C.POINTER(_Brute)]
    l.jo_brute_f64.restype = C.c_int


def _ptr(a, ctype):
    return a.ctypes.data_as(C.POINTER(ctype)) if a is not None else None


class _Problem:
    """Holds contiguous copies of the arrays and the ctypes struct."""

    def __init__(self, prob: dict):
        sfx = prob["dtype"]
        t = _T[sfx]
        self.sfx, self.t = sfx, t
        dt = t["np"]
        self.arrs = {k: np.ascontiguousarray(prob[k], dtype=dt) for k in
                     ("cycles", "bits", "alpha", "beta", "rate", "deadline", "local_freq", "gpu_freq")}
        self.arrs["t_free"] = (np.ascontiguousarray(prob["t_free"], dtype=dt)
                               if prob.get("t_free") is not None else None)
        for k in USER_KEYS:
            self.arrs[k] = (np.ascontiguousarray(prob[k], dtype=dt)
                            if prob.get(k) is not None else None)
        I = self.arrs["rate"].shape[0]
        self.I, self.N, self.L, self.K, self.J = I, prob["N"], prob["L"], prob["K"], prob["J"]
        assert self.arrs["rate"].shape == (I, self.N)
        assert self.arrs["deadline"].shape == (I, self.N)
        assert self.arrs["cycles"].shape == (I, self.L)
        assert self.arrs["bits"].shape == (I, self.L + 1)
        assert self.arrs["alpha"].shape == (I, self.L) and self.arrs["beta"].shape == (I, self.L)
        assert self.arrs["local_freq"].shape == (self.K,) and self.arrs["gpu_freq"].shape == (self.J,)
        for k in USER_KEYS:
            if self.arrs[k] is not None:
                want = (I, self.N, self.K) if k == "user_local_freq" else (I, self.N)
                assert self.arrs[k].shape == want, (k, self.arrs[k].shape, want)
        R = t["real"]
        self.s = t["problem"](I, self.N, self.L, self.K, self.J,
                              *[_ptr(self.arrs[k], R) for k in ("cycles", "bits", "alpha", "beta",
                                                                "rate", "deadline", "t_free",
                                                                "local_freq", "gpu_freq")],
                              float(prob["kappa"]), float(prob["p_tx"]), float(prob["gpu_c"]),
                              float(prob["gpu_p_static"]), int(prob.get("mode", 0)),
                              *[_ptr(self.arrs[k], R) for k in USER_KEYS])


def _chunks(n, parts):
    parts = max(1, min(parts, n))
    step = (n + parts - 1) // parts
    return [(a, min(step, n - a)) for a in range(0, n, step)]


# search variants (the JO_MODE_* bits of jdob_oracle.h)
MODE_GREEDY, MODE_FIXED_EDGE, MODE_BINARY, MODE_CONTINUOUS = 1, 2, 4, 8


def solve(prob: dict, threads: int = 1) -> dict:
    """Oracle policy of every instance of `prob` (see jdob_oracle.h); the
    search variant is ``prob.get("mode", 0)``."""
    P = _Problem(prob)
    l = lib()
    I, N, dt = P.I, P.N, P.t["np"]
    out = {"status": np.empty(I, np.int32), "cut": np.empty(I, np.int32),
           "gpu_level": np.empty(I, np.int32), "batch": np.empty(I, np.int32),
           "energy": np.empty(I, dt), "t_free_out": np.empty(I, dt),
           "user_level": np.empty((I, N), np.int8), "user_offload": np.empty((I, N), np.int8),
           "energy_second": np.empty(I, dt), "num_feasible": np.empty(I, np.int32),
           "num_user_evals": np.empty(I, np.int64), "user_freq": np.empty((I, N), dt)}
    R = P.t["real"]
    pol = P.t["policy"](*[_ptr(out[k], c) for k, c in (
        ("status", C.c_int32), ("cut", C.c_int32), ("gpu_level", C.c_int32), ("batch", C.c_int32),
        ("energy", R), ("t_free_out", R), ("user_level", C.c_int8), ("user_offload", C.c_int8),
        ("energy_second", R), ("num_feasible", C.c_int32), ("num_user_evals", C.c_int64),
        ("user_freq", R))])
    fn = getattr(l, "jo_solve_" + P.sfx)

    def run(ch):
        rc = fn(C.byref(P.s), ch[0], ch[1], C.byref(pol))
        if rc != 0:
            raise RuntimeError(f"jo_solve failed: {rc}")

    if I == 0:
        return out
    if threads <= 1:
        run((0, I))
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, _chunks(I, threads * 4)))
    return out


def solve_grouped(prob: dict, threads: int = 1) -> dict:
    """Outer grouping of every instance (jo_solve_grouped in jdob_oracle.h)."""
    P = _Problem(prob)
    l = lib()
    I, N, dt = P.I, P.N, P.t["np"]
    out = {"status": np.empty(I, np.int32), "num_groups": np.empty(I, np.int32),
           "energy": np.empty(I, dt), "t_free_out": np.empty(I, dt),
           "order": np.empty((I, N), np.int16), "group_end": np.empty((I, N), np.int16),
           "group_cut": np.empty((I, N), np.int32), "group_gpu_level": np.empty((I, N), np.int32),
           "group_batch": np.empty((I, N), np.int32), "group_energy": np.empty((I, N), dt),
           "group_t_free": np.empty((I, N), dt), "user_level": np.empty((I, N), np.int8),
           "user_offload": np.empty((I, N), np.int8), "user_group": np.empty((I, N), np.int8),
           "num_inner": np.empty(I, np.int64), "num_feasible": np.empty(I, np.int64),
           "num_user_evals": np.empty(I, np.int64), "user_freq": np.empty((I, N), dt)}
    R = P.t["real"]
    types = dict(status=C.c_int32, num_groups=C.c_int32, energy=R, t_free_out=R, order=C.c_int16,
                 group_end=C.c_int16, group_cut=C.c_int32, group_gpu_level=C.c_int32,
                 group_batch=C.c_int32, group_energy=R, group_t_free=R, user_level=C.c_int8,
                 user_offload=C.c_int8, user_group=C.c_int8, num_inner=C.c_int64,
                 num_feasible=C.c_int64, num_user_evals=C.c_int64, user_freq=R)
    g = P.t["grouped"](*[_ptr(out[k], types[k]) for k, _ in P.t["grouped"]._fields_])
    fn = getattr(l, "jo_solve_grouped_" + P.sfx)

    def run(ch):
        rc = fn(C.byref(P.s), ch[0], ch[1], C.byref(g))
        if rc != 0:
            raise RuntimeError(f"jo_solve_grouped failed: {rc}")

    if I == 0:
        return out
    if threads <= 1:
        run((0, I))
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, _chunks(I, threads * 4)))
    return out


def eval_grouping(prob: dict, inst: int, group_end, group_cut, group_gpu_level, group_batch) -> dict:
    """Chained evaluation of a given grouped policy of one instance."""
    P = _Problem(prob)
    G = len(group_end)
    ge = np.ascontiguousarray(group_end, np.int16)
    gc = np.ascontiguousarray(group_cut, np.int32)
    gj = np.ascontiguousarray(group_gpu_level, np.int32)
    gb = np.ascontiguousarray(group_batch, np.int32)
    ul = np.empty(P.N, np.int8)
    uo = np.empty(P.N, np.int8)
    uf = np.empty(P.N, P.t["np"])
    g = P.t["grouping"](G, _ptr(ge, C.c_int16), _ptr(gc, C.c_int32), _ptr(gj, C.c_int32),
                        _ptr(gb, C.c_int32), 0, 0, 0, _ptr(ul, C.c_int8), _ptr(uo, C.c_int8),
                        _ptr(uf, P.t["real"]))
    rc = getattr(lib(), "jo_eval_grouping_" + P.sfx)(C.byref(P.s), inst, C.byref(g))
    if rc != 0:
        raise RuntimeError(f"jo_eval_grouping failed: {rc}")
    return {"feasible": bool(g.feasible), "energy": g.energy, "t_free_out": g.t_free_out,
            "user_level": ul, "user_offload": uo, "user_freq": uf}


def user_tables(prob: dict) -> dict:
    P = _Problem(prob)
    I, N, L, dt = P.I, P.N, P.L, P.t["np"]
    out = {"order": np.empty((I, N), np.int16), "batch_deadline": np.empty((I, N), dt),
           "min_batch": np.empty(I, np.int32), "uplink_time": np.empty((I, L + 1, N), dt),
           "gamma": np.empty((I, L + 1, N), dt), "self_level": np.empty((I, L + 1, N), np.int8),
           "self_energy": np.empty((I, L + 1, N), dt), "self_slack": np.empty((I, L + 1, N), dt)}
    R = P.t["real"]
    tab = P.t["tables"](*[_ptr(out[k], c) for k, c in (
        ("order", C.c_int16), ("batch_deadline", R), ("min_batch", C.c_int32), ("uplink_time", R),
        ("gamma", R), ("self_level", C.c_int8), ("self_energy", R), ("self_slack", R))])
    rc = getattr(lib(), "jo_user_tables_" + P.sfx)(C.byref(P.s), 0, I, C.byref(tab))
    if rc != 0:
        raise RuntimeError(f"jo_user_tables failed: {rc}")
    return out


def eval_candidate(prob: dict, inst: int, s: int, j: int, b: int) -> dict:
    """One candidate; s == L is local computing (j, b ignored)."""
    P = _Problem(prob)
    ul = np.empty(P.N, np.int8)
    uo = np.empty(P.N, np.int8)
    uf = np.empty(P.N, P.t["np"])
    res = P.t["candidate"](0, 0, 0, 0, _ptr(ul, C.c_int8), _ptr(uo, C.c_int8),
                           _ptr(uf, P.t["real"]))
    rc = getattr(lib(), "jo_eval_candidate_" + P.sfx)(C.byref(P.s), inst, s, j, b, C.byref(res))
    if rc != 0:
        raise RuntimeError(f"jo_eval_candidate failed: {rc}")
    return {"feasible": bool(res.feasible), "energy": res.energy, "t_free_out": res.t_free_out,
            "gpu_latency": res.gpu_latency, "user_level": ul, "user_offload": uo,
            "user_freq": uf}


def brute(prob: dict, inst: int, suffix_only: bool) -> dict:
    """Exhaustive search (binary64 problems, tiny N and K only)."""
    P = _Problem(prob)
    assert P.sfx == "f64", "brute force takes binary64 problems"
    ul = np.empty(P.N, np.int8)
    uo = np.empty(P.N, np.int8)
    res = _Brute(0, 0.0, 0.0, 0, 0, 0, 0, _ptr(ul, C.c_int8), _ptr(uo, C.c_int8))
    rc = lib().jo_brute_f64(C.byref(P.s), inst, int(suffix_only), C.byref(res))
    if rc != 0:
        raise RuntimeError(f"jo_brute_f64 failed: {rc}")
    return {"found": bool(res.found), "energy": res.energy, "energy_second": res.energy_second,
            "cut": res.cut, "gpu_level": res.gpu_level, "batch": res.batch,
            "num_feasible": res.num_feasible, "user_level": ul, "user_offload": uo}
