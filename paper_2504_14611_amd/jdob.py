"""Thin ctypes binding of libjdob.so (include/jdob.h).

Argument marshalling only: every step of the evaluation runs in the HIP
kernels of the library.  PyTorch provides device memory and the stream.
There is no fallback: if the library is missing, loading raises.
"""

from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libjdob.so")

JDOB_F32, JDOB_F64 = 0, 1
JDOB_OK, JDOB_ERR_INVALID_ARG, JDOB_ERR_UNSUPPORTED, JDOB_ERR_HIP = 0, 1, 2, 3
# search mode bits (jdob_mode); a problem dict selects them with its "mode" key
JDOB_MODE_GRID, JDOB_MODE_GREEDY, JDOB_MODE_FIXED_EDGE_FREQ, JDOB_MODE_BINARY = 0, 1, 2, 4
JDOB_MODE_CONTINUOUS_CPU = 8

EXPORTS = ("jdob_eval_user_tables", "jdob_eval_joint", "jdob_solve_batch", "jdob_solve_grouped",
           "jdob_status_string")


class Problem(C.Structure):
    _fields_ = [("num_instances", C.c_int32), ("num_users", C.c_int32), ("num_layers", C.c_int32),
                ("num_local_levels", C.c_int32), ("num_gpu_levels", C.c_int32), ("dtype", C.c_int32),
                ("layer_cycles", C.c_void_p), ("out_bits", C.c_void_p), ("gpu_alpha", C.c_void_p),
                ("gpu_beta", C.c_void_p), ("uplink_rate", C.c_void_p), ("deadline", C.c_void_p),
                ("t_free", C.c_void_p), ("local_freq", C.c_void_p), ("gpu_freq", C.c_void_p),
                ("kappa", C.c_double), ("p_tx", C.c_double), ("gpu_c", C.c_double),
                ("gpu_p_static", C.c_double), ("mode", C.c_int32),
                ("user_zeta", C.c_void_p), ("user_kappa", C.c_void_p), ("user_p_tx", C.c_void_p),
                ("user_local_freq", C.c_void_p)]


class Policy(C.Structure):
    _fields_ = [("status", C.c_void_p), ("cut", C.c_void_p), ("gpu_level", C.c_void_p),
                ("batch", C.c_void_p), ("energy", C.c_void_p), ("t_free_out", C.c_void_p),
                ("user_level", C.c_void_p), ("user_offload", C.c_void_p),
                ("num_feasible", C.c_void_p), ("num_user_evals", C.c_void_p),
                ("user_freq", C.c_void_p)]


class UserTables(C.Structure):
    _fields_ = [("order", C.c_void_p), ("batch_deadline", C.c_void_p), ("min_batch", C.c_void_p),
                ("uplink_time", C.c_void_p), ("gamma", C.c_void_p), ("self_level", C.c_void_p),
                ("self_energy", C.c_void_p), ("self_slack", C.c_void_p)]


class GroupedPolicy(C.Structure):
    _fields_ = [(k, C.c_void_p) for k in (
        "status", "num_groups", "energy", "t_free_out", "order", "group_end", "group_cut",
        "group_gpu_level", "group_batch", "group_energy", "group_t_free", "user_level",
        "user_offload", "user_group", "num_inner", "num_feasible", "num_user_evals", "user_freq")]


_lib = None


def load(path: str = LIB_PATH):
    """Load libjdob.so; raises OSError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise OSError(f"{path} is missing: build it with "
                          "`python -c 'import __graft_entry__ as g; g.build()'`")
        lib = C.CDLL(path)
        lib.jdob_solve_batch.argtypes = [C.POINTER(Problem), C.POINTER(Policy), C.c_void_p]
        lib.jdob_eval_user_tables.argtypes = [C.POINTER(Problem), C.POINTER(UserTables), C.c_void_p]
        lib.jdob_eval_joint.argtypes = [C.POINTER(Problem), C.POINTER(UserTables), C.POINTER(Policy),
                                        C.c_void_p]
        lib.jdob_solve_grouped.argtypes = [C.POINTER(Problem), C.POINTER(GroupedPolicy), C.c_void_p]
        for f in ("jdob_solve_batch", "jdob_eval_user_tables", "jdob_eval_joint", "jdob_solve_grouped"):
            getattr(lib, f).restype = C.c_int
        lib.jdob_status_string.argtypes = [C.c_int]
        lib.jdob_status_string.restype = C.c_char_p
        _lib = lib
    return _lib


class JdobError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {load().jdob_status_string(code).decode()} ({code})")


def _check(code: int, where: str):
    if code != JDOB_OK:
        raise JdobError(code, where)


# ------------------------------------------------------------ device plumbing

# per-user parameters of heterogeneous users (optional): [I, N], levels [I, N, K]
USER_KEYS = ("user_zeta", "user_kappa", "user_p_tx", "user_local_freq")
_ARRAYS = ("cycles", "bits", "alpha", "beta", "rate", "deadline", "t_free", "local_freq",
           "gpu_freq") + USER_KEYS


def to_device(prob: dict, device="cuda") -> dict:
    """Copy the arrays of a generated problem to device tensors (torch)."""
    import torch
    out = {k: v for k, v in prob.items() if k not in _ARRAYS}
    for k in _ARRAYS:
        v = prob.get(k)
        out[k] = None if v is None else torch.from_numpy(np.ascontiguousarray(v)).to(device)
    return out


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def make_problem(d: dict) -> Problem:
    I = int(d["rate"].shape[0])
    return Problem(I, d["N"], d["L"], d["K"], d["J"], JDOB_F64 if d["dtype"] == "f64" else JDOB_F32,
                   _ptr(d["cycles"]), _ptr(d["bits"]), _ptr(d["alpha"]), _ptr(d["beta"]),
                   _ptr(d["rate"]), _ptr(d["deadline"]), _ptr(d.get("t_free")),
                   _ptr(d["local_freq"]), _ptr(d["gpu_freq"]),
                   float(d["kappa"]), float(d["p_tx"]), float(d["gpu_c"]), float(d["gpu_p_static"]),
                   int(d.get("mode", 0)), *[_ptr(d.get(k)) for k in USER_KEYS])


def _fdtype(d):
    import torch
    return torch.float64 if d["dtype"] == "f64" else torch.float32


def _want_freq(d: dict, freq: Optional[bool]) -> bool:
    """user_freq is allocated on request, by default only with a continuous
    CPU frequency (otherwise it is local_freq[user_level])."""
    return bool(int(d.get("mode", 0)) & JDOB_MODE_CONTINUOUS_CPU) if freq is None else freq


def alloc_policy(d: dict, counters: bool = True, freq: Optional[bool] = None) -> Dict[str, object]:
    import torch
    I, N = int(d["rate"].shape[0]), d["N"]
    dev = d["rate"].device
    i32 = dict(dtype=torch.int32, device=dev)
    out = {"status": torch.empty(I, **i32), "cut": torch.empty(I, **i32),
           "gpu_level": torch.empty(I, **i32), "batch": torch.empty(I, **i32),
           "energy": torch.empty(I, dtype=_fdtype(d), device=dev),
           "t_free_out": torch.empty(I, dtype=_fdtype(d), device=dev),
           "user_level": torch.empty((I, N), dtype=torch.int8, device=dev),
           "user_offload": torch.empty((I, N), dtype=torch.int8, device=dev),
           "num_feasible": torch.empty(I, **i32) if counters else None,
           "num_user_evals": torch.empty(I, dtype=torch.int64, device=dev) if counters else None,
           "user_freq": torch.empty((I, N), dtype=_fdtype(d), device=dev)
           if _want_freq(d, freq) else None}
    return out


def alloc_tables(d: dict) -> Dict[str, object]:
    import torch
    I, N, L = int(d["rate"].shape[0]), d["N"], d["L"]
    dev, ft = d["rate"].device, _fdtype(d)
    return {"order": torch.empty((I, N), dtype=torch.int16, device=dev),
            "batch_deadline": torch.empty((I, N), dtype=ft, device=dev),
            "min_batch": torch.empty(I, dtype=torch.int32, device=dev),
            "uplink_time": torch.empty((I, L + 1, N), dtype=ft, device=dev),
            "gamma": torch.empty((I, L + 1, N), dtype=ft, device=dev),
            "self_level": torch.empty((I, L + 1, N), dtype=torch.int8, device=dev),
            "self_energy": torch.empty((I, L + 1, N), dtype=ft, device=dev),
            "self_slack": torch.empty((I, L + 1, N), dtype=ft, device=dev)}


def alloc_grouped(d: dict, counters: bool = True, freq: Optional[bool] = None) -> Dict[str, object]:
    import torch
    I, N = int(d["rate"].shape[0]), d["N"]
    dev, ft = d["rate"].device, _fdtype(d)

    def t(shape, dtype):
        return torch.empty(shape, dtype=dtype, device=dev)
    out = {"status": t(I, torch.int32), "num_groups": t(I, torch.int32), "energy": t(I, ft),
           "t_free_out": t(I, ft), "order": t((I, N), torch.int16),
           "group_end": t((I, N), torch.int16), "group_cut": t((I, N), torch.int32),
           "group_gpu_level": t((I, N), torch.int32), "group_batch": t((I, N), torch.int32),
           "group_energy": t((I, N), ft), "group_t_free": t((I, N), ft),
           "user_level": t((I, N), torch.int8), "user_offload": t((I, N), torch.int8),
           "user_group": t((I, N), torch.int8)}
    for k in ("num_inner", "num_feasible", "num_user_evals"):
        out[k] = t(I, torch.int64) if counters else None
    out["user_freq"] = t((I, N), ft) if _want_freq(d, freq) else None
    return out


def make_policy(o: dict) -> Policy:
    return Policy(*[_ptr(o.get(k)) for k, _ in Policy._fields_])


def make_tables(t: dict) -> UserTables:
    return UserTables(*[_ptr(t.get(k)) for k, _ in UserTables._fields_])


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def solve_batch(d: dict, out: Optional[dict] = None, stream=None, counters: bool = True,
                freq: Optional[bool] = None) -> dict:
    """jdob_solve_batch on device tensors; returns the (device) output dict."""
    if out is None:
        out = alloc_policy(d, counters, freq)
    p, pol = make_problem(d), make_policy(out)
    _check(load().jdob_solve_batch(C.byref(p), C.byref(pol), _stream(stream)), "jdob_solve_batch")
    return out


def solve_grouped(d: dict, out: Optional[dict] = None, stream=None, counters: bool = True,
                  freq: Optional[bool] = None) -> dict:
    """jdob_solve_grouped on device tensors; returns the (device) output dict."""
    if out is None:
        out = alloc_grouped(d, counters, freq)
    p = make_problem(d)
    g = GroupedPolicy(*[_ptr(out.get(k)) for k, _ in GroupedPolicy._fields_])
    _check(load().jdob_solve_grouped(C.byref(p), C.byref(g), _stream(stream)), "jdob_solve_grouped")
    return out


def eval_user_tables(d: dict, out: Optional[dict] = None, stream=None) -> dict:
    if out is None:
        out = alloc_tables(d)
    p, tab = make_problem(d), make_tables(out)
    _check(load().jdob_eval_user_tables(C.byref(p), C.byref(tab), _stream(stream)),
           "jdob_eval_user_tables")
    return out


def eval_joint(d: dict, tables: dict, out: Optional[dict] = None, stream=None,
               counters: bool = True, freq: Optional[bool] = None) -> dict:
    if out is None:
        out = alloc_policy(d, counters, freq)
    p, tab, pol = make_problem(d), make_tables(tables), make_policy(out)
    _check(load().jdob_eval_joint(C.byref(p), C.byref(tab), C.byref(pol), _stream(stream)),
           "jdob_eval_joint")
    return out


def to_host(o: dict) -> dict:
    return {k: (None if v is None else v.cpu().numpy()) for k, v in o.items()}
