"""Pins of the oracle's continuous CPU frequency (oracle.MODE_CONTINUOUS; no
GPU needed).

Eq. (20) with its clamp: each user runs at the slowest frequency that meets
its budget, raised to f_min, within [local_freq[0], local_freq[K-1]].  Pinned
against:

* the exact-rational model, which solves each user's frequency in closed
  form (the energy kappa f^2 C grows with f), with every combination of the
  other mode bits;
* orderings that hold for any input: the continuous range contains every
  discrete level, so a continuous solve is feasible exactly when the
  discrete one is and never costs more; with denser levels the discrete
  energy falls towards the continuous one;
* the frequencies themselves: inside the range, and an offloader above
  f_min finishes its local part exactly at its budget.
"""

import numpy as np
import pytest

import oracle
from paper_2504_14611_amd import workloads as W
from tests import exact_model
from tests.test_oracle import tiny

CONT = oracle.MODE_CONTINUOUS


def with_mode(p, mode):
    q = dict(p)
    q["mode"] = mode
    return q


@pytest.mark.parametrize("extra", [0, 1, 2, 4, 5])
@pytest.mark.parametrize("stream", [860, 861])
def test_continuous_matches_exact_rational(extra, stream):
    p = with_mode(tiny(4, 4, 3, 3, 16, deadline=("per_user", 0.03, 0.4), stream=stream), CONT | extra)
    o = oracle.solve(p)
    for inst in range(16):
        ex = exact_model.solve_exact(p, inst, suffix_only=True)
        if ex is None:
            assert o["status"][inst] == 1, inst
            continue
        assert o["status"][inst] == 0, inst
        assert o["energy"][inst] == pytest.approx(float(ex["energy"]), rel=1e-12), inst
        gap = (ex["energy_second"] - ex["energy"]) / ex["energy"] if ex["energy_second"] else 1
        if gap > 1e-9:
            assert (o["cut"][inst], o["gpu_level"][inst], o["batch"][inst]) == \
                (ex["cut"], ex["gpu_level"], ex["batch"]), inst
            assert np.allclose(o["user_freq"][inst], [float(x) for x in ex["levels"]], rtol=1e-13)
            assert o["t_free_out"][inst] == pytest.approx(float(ex["t_free_out"]), rel=1e-12)
            assert (o["user_level"][inst] == -1).all()


def test_continuous_pin_is_sensitive():
    """On the pin's inputs frequencies strictly inside the range occur for
    offloaders and for local users, and continuous beats the levels."""
    p = tiny(4, 4, 3, 3, 16, deadline=("per_user", 0.03, 0.4), stream=860)
    c, d = oracle.solve(with_mode(p, CONT)), oracle.solve(p)
    f = c["status"] == 0
    lo, hi = p["local_freq"][0], p["local_freq"][-1]
    inside = (c["user_freq"][f] > lo) & (c["user_freq"][f] < hi)
    assert (inside & (c["user_offload"][f] == 1)).sum() > 3
    assert (inside & (c["user_offload"][f] == 0)).sum() > 3
    assert (c["energy"][f] < d["energy"][f]).sum() >= 5


@pytest.mark.parametrize("name,n", [("c1", 512), ("c2b", 256), ("p4a", 256), ("p4b", 128),
                                    ("c4b", 8)])
def test_continuous_never_costs_more_than_levels(name, n):
    p = W.generate(W.WORKLOADS[name], 0, n)
    c = oracle.solve(with_mode(p, CONT), threads=4)
    d = oracle.solve(with_mode(p, 0), threads=4)
    assert np.array_equal(c["status"], d["status"])
    f = c["status"] == 0
    assert (c["energy"][f] <= d["energy"][f] * (1 + 2e-6)).all()
    assert (c["num_feasible"] == d["num_feasible"]).all()   # the same tests decide feasibility


def test_dense_levels_approach_continuous():
    p = W.generate(W.WORKLOADS["p4a"], 0, 64)
    p["dtype"] = "f64"
    for k in ("cycles", "bits", "alpha", "beta", "rate", "deadline", "t_free", "local_freq", "gpu_freq"):
        p[k] = p[k].astype(np.float64)
    c = oracle.solve(with_mode(p, CONT))
    q = with_mode(p, 0)
    q["K"] = 1025
    q["local_freq"] = np.linspace(p["local_freq"][0], p["local_freq"][-1], 1025)
    d = oracle.solve(q)
    f = c["status"] == 0
    assert np.array_equal(c["status"], d["status"])
    rel = d["energy"][f] / c["energy"][f] - 1
    assert (rel >= -1e-12).all() and rel.max() < 2e-3


def test_frequencies_in_range_and_tight():
    p = W.generate(W.WORKLOADS["p4a"], 0, 128)
    o = oracle.solve(p)
    lo, hi = p["local_freq"][0], p["local_freq"][-1]
    L, J, N = p["L"], p["J"], p["N"]
    for inst in np.nonzero(o["status"] == 0)[0][:64]:
        fr = o["user_freq"][inst]
        assert ((fr >= lo) & (fr <= hi)).all()
        s, j, b = o["cut"][inst], o["gpu_level"][inst], o["batch"][inst]
        if s == L:
            continue
        C = np.float64(p["cycles"][inst, :s].astype(np.float64).sum())
        phi = (p["alpha"][inst, s:].astype(np.float64).sum()
               + p["beta"][inst, s:].astype(np.float64).sum() * b) * p["gpu_freq"][-1] / p["gpu_freq"][j]
        off = o["user_offload"][inst] == 1
        lo_b = p["deadline"][inst][off].min()
        for m in np.nonzero(off)[0]:
            budget = lo_b - phi - p["bits"][inst, s] / p["rate"][inst, m]
            assert C / fr[m] <= budget * (1 + 1e-5)            # meets (7)
            if fr[m] > lo * (1 + 1e-6) and C > 0:
                assert C / fr[m] == pytest.approx(budget, rel=1e-4)   # and no slower
