"""Seeded synthetic J-DOB workloads (input generation only).

Every random number is a counter-based draw: the n-th output of a SplitMix64
stream (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014) whose seed is hashed from (seed, workload, field).
The counter is ``instance * 4096 + index + 1``, so any slice of instances can
be regenerated on its own and the result does not depend on the order of
generation.  u = top 53 bits * 2**-53 is uniform on [0, 1).

Values are drawn in binary64 and rounded once to the workload's precision.
This module contains no arithmetic of the method: it only produces the
arrays of the system model of Sec. II (layer cycles, output bits, GPU batch
latency coefficients, uplink rates, deadlines, frequency levels).

Workload recipes (units SI; LU = log-uniform, U = uniform):

  name  I          N    L   K   J   precision
  c0    256        4    8   4   4   f64   cycles LU[1e7,1e9], bits LU[1e4,1e6],
                                          one deadline per instance U[50,500] ms
  c1    4096       8    16  8   8   f32   as c0, per-user deadlines U[50,500] ms
  c2    65536      16   22  16  16  f32   conv-then-FC: cycles LU[1e6,1e7] for
                                          layers 1..L-2 and LU[1e5,1e6] for the
                                          last two; bits 4e6 * 0.7**(l-1);
                                          one deadline per instance U[30,300] ms
  c3    1048576    32   22  16  32  f32   as c2; rates U[1,100] Mbit/s;
                                          per-user deadlines U[30,500] ms
  c4    262144     128  50  32  64  f32   cycles LU[1e6,5e8], bits LU[1e3,4e6];
                                          per-user deadline, a fair coin picks
                                          U[20,80] ms or U[200,800] ms
Common: O_0 = 1e6 input bits; alpha_l LU[0.1,2] ms, beta_l LU[0.05,1] ms;
rates U[5,50] Mbit/s unless stated; CPU levels evenly spaced over
[0.5,2.0] GHz, GPU levels over [0.8,2.0] GHz (endpoints included);
kappa = 1e-28, p_tx = 0.5 W, GPU power gpu_c*g^3 + 50 W with
gpu_c = 3.125e-26 W/Hz^3; t_free = 0.  Seeds: 0 for c0, the workload index
for c1..c4.

Outer-grouping workloads (the paper's different-deadline experiments):

  g10   65536      10   22  16  32  f32   c3's layer profile and rates;
  g20   32768      20   22  16  32  f32   deadline T_m = (1 + beta_m) * (sum of
                                          the cycles) / top CPU level, beta_m
                                          U[0,10]; kappa = 2.25e-26 (device
                                          power at 2 GHz = 0.6 x GPU power at
                                          2 GHz)

Paper-parameter workloads p4a, p4b, p5 (Table I, continuous CPU frequency)
are described where they are defined below.

Heterogeneous users (per-user zeta_m, kappa_m, p_m and CPU range, Sec. II):

  h1    262144     16   22  8   32  f32   c3's layers and rates; zeta_m
                                          LU[0.5,2], kappa_m = 2.25e-26 x
                                          LU[0.5,2], p_m U[0.2,1] W, levels
                                          from U[0.3,0.8] to U[1.5,2.5] GHz;
                                          T_m = (1 + beta_m) x the user's own
                                          local latency at its top level,
                                          beta_m U[0.5,4]
  h2    65536      10   8   2   64  f32   p4a with zeta_m LU[0.8,1.25],
                                          kappa_m x LU[0.5,2], p_m U[0.5,1.5] W,
                                          continuous range [U[1.2,1.8],
                                          U[2.2,3.0]] GHz, beta_m U[0.5,5]
  h5    65536      10   8   2   64  f32   h2 with beta_m U[0,10], solved with
                                          the outer grouping

Companion workloads exist only to widen parity coverage: ``c2b`` (c2 with
conv-layer cycles LU[1e6,1e8], many offloading winners) and ``c4b`` (c4
shapes with layer cycles LU[3e5,3e6] and alpha, beta scaled by 0.005, so that
every instance is feasible and batches of 70-128 users win).
"""

from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Tuple

import numpy as np

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

FIELD_CYCLES = 1
FIELD_BITS = 2
FIELD_ALPHA = 3
FIELD_BETA = 4
FIELD_RATE = 5
FIELD_DEADLINE = 6
FIELD_DEADLINE_MODE = 7
FIELD_ZETA = 8
FIELD_KAPPA = 9
FIELD_PTX = 10
FIELD_FMIN = 11
FIELD_FMAX = 12


def _mix64(z: np.ndarray) -> np.ndarray:
    """SplitMix64 output function (the variant with shifts 30, 27, 31)."""
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def stream_seed(seed: int, stream: int, field: int) -> np.uint64:
    key = np.array([(seed << 32) ^ (stream << 16) ^ field], dtype=np.uint64)
    return _mix64(key)[0]


def uniform01(seed: int, stream: int, field: int, inst: np.ndarray,
              idx: np.ndarray) -> np.ndarray:
    """u in [0,1) for every (instance, index) pair (broadcasting arrays)."""
    base = stream_seed(seed, stream, field)
    ctr = (inst.astype(np.uint64) * np.uint64(4096)
           + idx.astype(np.uint64) + np.uint64(1))
    with np.errstate(over="ignore"):
        z = _mix64(base + ctr * _GOLDEN)
    return (z >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)


def _lu(u, lo, hi):
    return np.exp(np.log(lo) + u * (np.log(hi) - np.log(lo)))


def _u(u, lo, hi):
    return lo + u * (hi - lo)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    stream: int
    seed: int
    num_instances: int
    N: int
    L: int
    K: int
    J: int
    dtype: str                      # "f32" or "f64"
    cycles: Tuple                   # ("lu", lo, hi) or ("convfc", conv_lo, conv_hi, fc_lo, fc_hi, n_fc)
    bits: Tuple                     # ("lu", lo, hi) or ("geom", first, ratio)
    rate: Tuple = ("u", 5e6, 50e6)
    deadline: Tuple = ("per_user", 0.05, 0.5)   # or ("shared", lo, hi) / ("bimodal", lo1, hi1,
                                                # lo2, hi2) / ("beta", lo, hi): T = (1 + beta) *
                                                # local latency at the top CPU level
    alpha: Tuple = ("lu", 1e-4, 2e-3)
    beta: Tuple = ("lu", 5e-5, 1e-3)
    input_bits: float = 1e6
    local_f: Tuple = (0.5e9, 2.0e9)
    gpu_f: Tuple = (0.8e9, 2.0e9)
    kappa: float = 1e-28
    p_tx: float = 0.5
    gpu_c: float = 3.125e-26
    gpu_p_static: float = 50.0
    gpu_scale: float = 1.0          # multiplies alpha and beta (companions only)
    mode: int = 0                   # search mode the workload is solved with
    users: Optional[Tuple] = None   # heterogeneous users: ("hetero", zeta_lo, zeta_hi,
                                    # kappa_mult_lo, kappa_mult_hi, ptx_lo, ptx_hi,
                                    # fmin_lo, fmin_hi, fmax_lo, fmax_hi)

    def np_dtype(self):
        return np.float64 if self.dtype == "f64" else np.float32

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    "c0": Workload("c0", 0, 0, 256, 4, 8, 4, 4, "f64",
                   cycles=("lu", 1e7, 1e9), bits=("lu", 1e4, 1e6),
                   deadline=("shared", 0.05, 0.5)),
    "c1": Workload("c1", 1, 1, 4096, 8, 16, 8, 8, "f32",
                   cycles=("lu", 1e7, 1e9), bits=("lu", 1e4, 1e6),
                   deadline=("per_user", 0.05, 0.5)),
    "c2": Workload("c2", 2, 2, 65536, 16, 22, 16, 16, "f32",
                   cycles=("convfc", 1e6, 1e7, 1e5, 1e6, 2),
                   bits=("geom", 4e6, 0.7),
                   deadline=("shared", 0.03, 0.3)),
    "c3": Workload("c3", 3, 3, 1048576, 32, 22, 16, 32, "f32",
                   cycles=("convfc", 1e6, 1e7, 1e5, 1e6, 2),
                   bits=("geom", 4e6, 0.7),
                   rate=("u", 1e6, 100e6),
                   deadline=("per_user", 0.03, 0.5)),
    "c4": Workload("c4", 4, 4, 262144, 128, 50, 32, 64, "f32",
                   cycles=("lu", 1e6, 5e8), bits=("lu", 1e3, 4e6),
                   deadline=("bimodal", 0.02, 0.08, 0.2, 0.8)),
}
# Outer grouping (different deadlines, as in the paper's Sec. IV-B): 10 and
# 20 users, deadlines from beta in [0, 10], the layer profile of c3, and a
# device whose power at its top frequency is 0.6 of the GPU's at its top
# frequency (kappa * f^3 = 0.6 * (gpu_c * g^3 + P0), the eta of Table I).
WORKLOADS["g10"] = Workload("g10", 5, 5, 65536, 10, 22, 16, 32, "f32",
                            cycles=("convfc", 1e6, 1e7, 1e5, 1e6, 2),
                            bits=("geom", 4e6, 0.7), rate=("u", 1e6, 100e6),
                            deadline=("beta", 0.0, 10.0), kappa=2.25e-26)
WORKLOADS["g20"] = WORKLOADS["g10"].replace(name="g20", stream=6, seed=6, num_instances=32768, N=20)
# The paper's own parameters (Table I, Sec. IV) with a synthetic
# MobileNetV2-like chain of 8 blocks (the block profile itself is not in the
# paper's text): a 224x224x3 8-bit input, block outputs shrinking from
# 1.6 Mbit by 0.6 per block, block cycles LU[0.5e6, 1.6e6] (about 3.2 ms of
# local inference at 2.6 GHz); the edge's batch-1 latency equals the local
# latency at the top frequencies (alpha_m = 1 of Table I), 0.8 + 0.2 b of it
# at batch b; uplink 10 MHz * log2(1 + 10^3) for every user (SNR 30 dB),
# p_u = 1 W; CPU frequency continuous in [1.5, 2.6] GHz; GPU levels every
# rho = 0.03 GHz from 0.21 to 2.1 GHz; device power 0.6 of the edge's at the
# top frequencies (eta_m = 0.6: 180 W vs 300 W), edge energy proportional to
# f_e^2 (no static power).
_R_TABLE_I = 10e6 * float(np.log2(1.0 + 1e3))
WORKLOADS["p4a"] = Workload("p4a", 7, 7, 65536, 10, 8, 2, 64, "f32",
                            cycles=("lu", 0.5e6, 1.6e6), bits=("geom", 1.6e6, 0.6),
                            rate=("u", _R_TABLE_I, _R_TABLE_I),
                            deadline=("beta", 2.13, 2.13),
                            alpha=("per_cycle", 0.8, 2.6e9), beta=("per_cycle", 0.2, 2.6e9),
                            input_bits=224 * 224 * 3 * 8.0,
                            local_f=(1.5e9, 2.6e9), gpu_f=(0.21e9, 2.1e9),
                            kappa=180.0 / 2.6e9 ** 3, p_tx=1.0,
                            gpu_c=300.0 / 2.1e9 ** 3, gpu_p_static=0.0, mode=8)
WORKLOADS["p4b"] = WORKLOADS["p4a"].replace(name="p4b", stream=8, seed=8,
                                            deadline=("beta", 30.25, 30.25))
WORKLOADS["p5"] = WORKLOADS["p4a"].replace(name="p5", stream=9, seed=9,
                                           deadline=("beta", 0.0, 10.0))
# Heterogeneous users (Sec. II: zeta_m, kappa_m, p_m and the CPU frequency
# range differ per device): h1 with 8 levels per user, h2 with the Table I
# setup of p4a and a continuous frequency in each user's own range.
WORKLOADS["h1"] = Workload("h1", 15, 15, 262144, 16, 22, 8, 32, "f32",
                           cycles=("convfc", 1e6, 1e7, 1e5, 1e6, 2),
                           bits=("geom", 4e6, 0.7), rate=("u", 1e6, 100e6),
                           deadline=("beta", 0.5, 4.0), kappa=2.25e-26,
                           users=("hetero", 0.5, 2.0, 0.5, 2.0, 0.2, 1.0, 0.3e9, 0.8e9,
                                  1.5e9, 2.5e9))
WORKLOADS["h2"] = WORKLOADS["p4a"].replace(name="h2", stream=16, seed=16,
                                           deadline=("beta", 0.5, 5.0),
                                           users=("hetero", 0.8, 1.25, 0.5, 2.0, 0.5, 1.5,
                                                  1.2e9, 1.8e9, 2.2e9, 3.0e9))
# the outer grouping with heterogeneous users: h2 with deadlines from beta_m in
# [0, 10] (p5's spread)
WORKLOADS["h5"] = WORKLOADS["h2"].replace(name="h5", stream=17, seed=17,
                                          deadline=("beta", 0.0, 10.0))
WORKLOADS["c2b"] = WORKLOADS["c2"].replace(
    name="c2b", stream=12, cycles=("convfc", 1e6, 1e8, 1e5, 1e6, 2))
WORKLOADS["c4b"] = WORKLOADS["c4"].replace(
    name="c4b", stream=14, cycles=("lu", 3e5, 3e6), gpu_scale=0.005)


def levels(lo: float, hi: float, n: int) -> np.ndarray:
    if n == 1:
        return np.array([hi], dtype=np.float64)
    return lo + np.arange(n, dtype=np.float64) * ((hi - lo) / (n - 1))


def generate(w: Workload, start: int = 0, count: Optional[int] = None) -> dict:
    """Arrays of instances [start, start+count) of workload `w`.

    Returns a dict with keys cycles [I,L], bits [I,L+1], alpha [I,L],
    beta [I,L], rate [I,N], deadline [I,N], t_free [I], local_freq [K],
    gpu_freq [J] (all in the workload's precision) and the scalars kappa,
    p_tx, gpu_c, gpu_p_static plus N, L, K, J, dtype.
    """
    if count is None:
        count = w.num_instances - start
    N, L = w.N, w.L
    inst = np.arange(start, start + count, dtype=np.int64)[:, None]
    lidx = np.arange(L, dtype=np.int64)[None, :]
    midx = np.arange(N, dtype=np.int64)[None, :]
    s, st = w.seed, w.stream

    # layer cycles
    u = uniform01(s, st, FIELD_CYCLES, inst, lidx)
    if w.cycles[0] == "lu":
        cycles = _lu(u, w.cycles[1], w.cycles[2])
    elif w.cycles[0] == "convfc":
        _, clo, chi, flo, fhi, nfc = w.cycles
        conv = np.broadcast_to(lidx < L - nfc, u.shape)
        cycles = np.where(conv, _lu(u, clo, chi), _lu(u, flo, fhi))
    else:
        raise ValueError(w.cycles)

    # output bits O_0 .. O_L
    bits = np.empty((count, L + 1), dtype=np.float64)
    bits[:, 0] = w.input_bits
    if w.bits[0] == "lu":
        bits[:, 1:] = _lu(uniform01(s, st, FIELD_BITS, inst, lidx), w.bits[1], w.bits[2])
    elif w.bits[0] == "geom":
        bits[:, 1:] = w.bits[1] * w.bits[2] ** np.arange(L, dtype=np.float64)[None, :]
    else:
        raise ValueError(w.bits)

    if w.alpha[0] == "per_cycle":
        # batch latency of layer l at the top GPU level: (a + b * batch) times
        # the layer's local latency at the top CPU level
        t_l = cycles / w.alpha[2]
        alpha, beta = w.alpha[1] * t_l, w.beta[1] * t_l
    else:
        alpha = _lu(uniform01(s, st, FIELD_ALPHA, inst, lidx), *w.alpha[1:]) * w.gpu_scale
        beta = _lu(uniform01(s, st, FIELD_BETA, inst, lidx), *w.beta[1:]) * w.gpu_scale
    rate = _u(uniform01(s, st, FIELD_RATE, inst, midx), *w.rate[1:])

    users = None
    if w.users is not None:
        # Sec. II: per-user cycles per unit of work, switched capacitance,
        # transmit power and CPU frequency range (K levels evenly spaced)
        _, z0, z1, k0, k1, p0, p1, fl0, fl1, fh0, fh1 = w.users
        zeta = _lu(uniform01(s, st, FIELD_ZETA, inst, midx), z0, z1)
        kap = w.kappa * _lu(uniform01(s, st, FIELD_KAPPA, inst, midx), k0, k1)
        ptx = _u(uniform01(s, st, FIELD_PTX, inst, midx), p0, p1)
        fmin = _u(uniform01(s, st, FIELD_FMIN, inst, midx), fl0, fl1)
        fmax = _u(uniform01(s, st, FIELD_FMAX, inst, midx), fh0, fh1)
        if w.K == 1:
            lf = fmax[:, :, None]
        else:
            step = (fmax - fmin) / (w.K - 1)
            lf = fmin[:, :, None] + np.arange(w.K, dtype=np.float64)[None, None, :] * step[:, :, None]
        users = dict(user_zeta=zeta, user_kappa=kap, user_p_tx=ptx, user_local_freq=lf)

    kind = w.deadline[0]
    if kind == "shared":
        d = _u(uniform01(s, st, FIELD_DEADLINE, inst, np.zeros((1, 1), np.int64)),
               w.deadline[1], w.deadline[2])
        deadline = np.broadcast_to(d, (count, N)).copy()
    elif kind == "per_user":
        deadline = _u(uniform01(s, st, FIELD_DEADLINE, inst, midx), w.deadline[1], w.deadline[2])
    elif kind == "bimodal":
        _, a1, b1, a2, b2 = w.deadline
        u = uniform01(s, st, FIELD_DEADLINE, inst, midx)
        first = uniform01(s, st, FIELD_DEADLINE_MODE, inst, midx) < 0.5
        deadline = np.where(first, _u(u, a1, b1), _u(u, a2, b2))
    elif kind == "beta":
        # Sec. IV: beta_m = T_m / (local latency of the whole DNN at the top
        # CPU frequency) - 1, drawn uniformly in [lo, hi]
        beta_m = _u(uniform01(s, st, FIELD_DEADLINE, inst, midx), w.deadline[1], w.deadline[2])
        if users is None:
            t_local = cycles.sum(axis=1, keepdims=True) / w.local_f[1]
        else:  # each user's own latency at its top frequency
            t_local = users["user_zeta"] * cycles.sum(axis=1, keepdims=True) / fmax
        deadline = (1.0 + beta_m) * t_local
    else:
        raise ValueError(w.deadline)

    dt = w.np_dtype()
    extra = {} if users is None else {k: np.ascontiguousarray(v, dtype=dt) for k, v in users.items()}
    return {**extra,
        "cycles": np.ascontiguousarray(cycles, dtype=dt),
        "bits": np.ascontiguousarray(bits, dtype=dt),
        "alpha": np.ascontiguousarray(alpha, dtype=dt),
        "beta": np.ascontiguousarray(beta, dtype=dt),
        "rate": np.ascontiguousarray(rate, dtype=dt),
        "deadline": np.ascontiguousarray(deadline, dtype=dt),
        "t_free": np.zeros(count, dtype=dt),
        "local_freq": levels(*w.local_f, w.K).astype(dt),
        "gpu_freq": levels(*w.gpu_f, w.J).astype(dt),
        "kappa": w.kappa, "p_tx": w.p_tx, "gpu_c": w.gpu_c,
        "gpu_p_static": w.gpu_p_static,
        "N": N, "L": L, "K": w.K, "J": w.J, "dtype": w.dtype, "mode": w.mode,
    }


def take(prob: dict, idx) -> dict:
    """Sub-batch of a generated problem (instance selection by index array)."""
    out = dict(prob)
    for k in ("cycles", "bits", "alpha", "beta", "rate", "deadline", "t_free") + USER_KEYS:
        if prob.get(k) is not None:
            out[k] = np.ascontiguousarray(prob[k][idx])
    return out


# per-user arrays of heterogeneous users: [I, N] and, for the levels, [I, N, K]
USER_KEYS = ("user_zeta", "user_kappa", "user_p_tx", "user_local_freq")


def num_instances(prob: dict) -> int:
    return int(prob["rate"].shape[0])
