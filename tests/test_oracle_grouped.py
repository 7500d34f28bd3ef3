"""Pins of the oracle's outer grouping (no GPU needed).

The paper's outer module groups users by deadline and calls the inner
algorithm once per group (Sec. II, Sec. IV-B); the grouping dynamic program
comes from its reference [9] and is not given, so the oracle implements the
reading stated in jdob_oracle.h: consecutive groups in deadline order, served
in that order, the GPU free time chained through Eq. (22), a front of
(energy, release) states per prefix, none dominated by another.  Pinned
against:

* an exact-rational version of the same dynamic program over the exact
  inner enumeration (tests/exact_model.py), which shares no code with it;
* brute force over every partition into consecutive groups, each evaluated
  with its release times chained: the program equals it on every instance
  of the pin (including Table-I inputs where keeping one state per prefix
  misses the optimum on half the instances);
* the chained re-evaluation of the oracle's own answer (jo_eval_grouping);
* closed cases: one user; the single group is one of the program's choices.
"""

import itertools

import numpy as np
import pytest

import oracle
from paper_2504_14611_amd import workloads as W
from tests import exact_model
from tests.test_oracle import tiny


def og_tiny(N, L, K, J, n, stream, kappa=4e-25, cycles=("lu", 1e6, 1e7),
            deadline=("beta", 0.0, 10.0), **kw):
    """Tiny grouping instances where several groups, some offloading, win on
    about half the instances (a costly device, cheap enough layers)."""
    w = W.WORKLOADS["g10"].replace(name="tiny_og", stream=stream, num_instances=n, N=N, L=L,
                                   K=K, J=J, dtype="f64", deadline=deadline, kappa=kappa,
                                   cycles=cycles, **kw)
    return W.generate(w)


def group_arrays(o, inst):
    G = int(o["num_groups"][inst])
    return (o["group_end"][inst, :G], o["group_cut"][inst, :G], o["group_gpu_level"][inst, :G],
            o["group_batch"][inst, :G])


@pytest.mark.parametrize("shape,stream", [((3, 3, 2, 3), 810), ((4, 3, 3, 2), 811), ((4, 2, 2, 3), 812)])
def test_grouped_matches_exact_rational(shape, stream):
    N, L, K, J = shape
    p = og_tiny(N, L, K, J, 10, stream)
    o = oracle.solve_grouped(p)
    for inst in range(10):
        ex = exact_model.solve_grouped_exact(p, inst)
        if ex is None:
            assert o["status"][inst] == 1
            continue
        assert o["status"][inst] == 0
        assert o["energy"][inst] == pytest.approx(float(ex["energy"]), rel=1e-12), inst
        assert o["t_free_out"][inst] == pytest.approx(float(ex["t_free_out"]), rel=1e-12, abs=1e-15)


def test_grouped_pin_is_sensitive():
    """On the pin's inputs the grouping matters: several groups, offloading
    groups and t_free chaining all occur."""
    groups, offl = [], 0
    for shape, stream in (((3, 3, 2, 3), 810), ((4, 3, 3, 2), 811), ((4, 2, 2, 3), 812)):
        p = og_tiny(*shape, 10, stream)
        o = oracle.solve_grouped(p)
        groups += list(o["num_groups"])
        offl += int((o["group_cut"][o["group_cut"] >= 0] < shape[1]).sum())
    assert max(groups) >= 2 and offl >= 5


def _partitions(N):
    """Every split of 0..N into consecutive groups, as lists of end points."""
    for cuts in itertools.product((0, 1), repeat=N - 1):
        yield [i + 1 for i in range(N - 1) if cuts[i]] + [N]


def _candidate(prob, inst, members, tfree, cand):
    """One candidate (cut, GPU level, batch) of the group `members` with the
    GPU free at tfree (cut == L: local computing)."""
    s, j, b = cand
    sub = _sub(prob, inst, members, tfree)
    return oracle.eval_candidate(sub, 0, s, max(j, 0), b)


def _single(prob, inst, members, tfree):
    return oracle.solve(_sub(prob, inst, members, tfree))


def _sub(prob, inst, members, tfree):
    sub = {k: prob[k] for k in ("local_freq", "gpu_freq", "kappa", "p_tx", "gpu_c",
                                 "gpu_p_static", "K", "J", "L", "dtype")}
    sub["mode"] = prob.get("mode", 0)
    sub["N"] = len(members)
    for k in ("cycles", "bits", "alpha", "beta"):
        sub[k] = np.ascontiguousarray(prob[k][inst:inst + 1])
    sub["rate"] = np.ascontiguousarray(prob["rate"][inst:inst + 1, members])
    sub["deadline"] = np.ascontiguousarray(prob["deadline"][inst:inst + 1, members])
    sub["t_free"] = np.array([tfree], prob["rate"].dtype)
    for k in oracle.USER_KEYS:  # heterogeneous users: the members' own parameters
        if prob.get(k) is not None:
            sub[k] = np.ascontiguousarray(prob[k][inst:inst + 1, members])
    return sub


def brute_force_grouping(p, inst):
    """Lowest total energy over every partition of the deadline order into
    consecutive groups, each group one inner solve with the GPU free at the
    previous group's release time (group results cached per (group, t_free))."""
    N = p["N"]
    T = p["deadline"]
    order = sorted(range(N), key=lambda m: (T[inst, m], m))
    cache = {}
    best = np.inf
    for ends in _partitions(N):
        tf, total, a = p["t_free"][inst], 0.0, 0
        for b in ends:
            key = (a, b, float(tf))
            if key not in cache:
                r = _single(p, inst, sorted(order[a:b]), tf)
                cache[key] = None if r["status"][0] != 0 else (float(r["energy"][0]), r["t_free_out"][0])
            if cache[key] is None:
                total = np.inf
                break
            total += cache[key][0]
            tf = cache[key][1]
            a = b
        best = min(best, total)
    return best


@pytest.mark.parametrize("name,n,N", [("g10", 12, 6), ("g10", 8, 7), ("p5", 16, 6), ("h5", 8, 5)])
def test_grouped_equals_brute_force_over_partitions(name, n, N):
    w = W.WORKLOADS[name].replace(N=N, num_instances=n, stream=820 + N + 7 * (name != "g10"))
    p = W.generate(w)
    o = oracle.solve_grouped(p)
    for inst in range(n):
        best = brute_force_grouping(p, inst)
        assert o["status"][inst] == (0 if np.isfinite(best) else 1)
        if np.isfinite(best):
            assert float(o["energy"][inst]) == pytest.approx(best, rel=1e-6), inst


def test_one_state_per_prefix_would_miss():
    """The inputs of the pin need the fronts: the program restricted to the
    lowest-energy state of every prefix misses the brute-force optimum on
    some of its p5 instances (so the equality above is not vacuous)."""
    w = W.WORKLOADS["p5"].replace(N=6, num_instances=16, stream=833)
    p = W.generate(w)
    misses = 0
    for inst in range(16):
        T = p["deadline"]
        order = sorted(range(6), key=lambda m: (T[inst, m], m))
        dp = {0: (0.0, p["t_free"][inst])}
        for i in range(1, 7):
            cands = []
            for j in range(i):
                if j not in dp:
                    continue
                r = _single(p, inst, sorted(order[j:i]), dp[j][1])
                if r["status"][0] == 0:
                    cands.append((dp[j][0] + float(r["energy"][0]), float(r["t_free_out"][0])))
            if cands:
                dp[i] = min(cands)
        misses += dp[6][0] > brute_force_grouping(p, inst) * (1 + 1e-6)
    assert misses >= 3


@pytest.mark.parametrize("name,n", [("g10", 64), ("g20", 16), ("c1", 128)])
def test_grouped_answer_reevaluates_bitwise(name, n):
    p = W.generate(W.WORKLOADS[name], 0, n)
    o = oracle.solve_grouped(p, threads=4)
    for inst in range(n):
        if o["status"][inst] != 0:
            continue
        ev = oracle.eval_grouping(p, inst, *group_arrays(o, inst))
        assert ev["feasible"]
        G = int(o["num_groups"][inst])
        # energies are summed group by group in both, so they agree bitwise
        assert ev["energy"] == o["energy"][inst]
        assert ev["t_free_out"] == o["t_free_out"][inst]
        assert np.array_equal(ev["user_level"], o["user_level"][inst])
        assert np.array_equal(ev["user_offload"], o["user_offload"][inst])
        ends = o["group_end"][inst, :G]
        assert ends[-1] == p["N"] and (np.diff(ends) > 0).all()
        # every user belongs to the group its deadline rank falls in
        rank = np.empty(p["N"], int)
        rank[o["order"][inst]] = np.arange(p["N"])
        assert np.array_equal(o["user_group"][inst], np.searchsorted(ends, rank, side="right"))


@pytest.mark.parametrize("name,n", [("g10", 128), ("c1", 256), ("c2b", 64)])
def test_grouped_never_worse_than_one_group(name, n):
    p = W.generate(W.WORKLOADS[name], 0, n)
    o = oracle.solve_grouped(p, threads=4)
    s = oracle.solve(p, threads=4)
    one = s["status"] == 0
    assert (o["status"][one] == 0).all()
    assert (o["energy"][one] <= s["energy"][one]).all()


def test_grouped_single_user_is_the_inner_solve():
    p = tiny(1, 6, 5, 4, 64, deadline=("per_user", 0.02, 0.3))
    o, s = oracle.solve_grouped(p), oracle.solve(p)
    assert np.array_equal(o["status"], s["status"])
    f = s["status"] == 0
    assert np.array_equal(o["energy"][f], s["energy"][f])
    assert np.array_equal(o["t_free_out"][f], s["t_free_out"][f])
    assert (o["num_groups"][f] == 1).all()
    assert np.array_equal(o["group_cut"][f, 0], s["cut"][f])
    assert np.array_equal(o["user_level"][f], s["user_level"][f])


def test_grouped_deadline_order_and_counters():
    p = W.generate(W.WORKLOADS["g10"], 0, 32)
    o = oracle.solve_grouped(p)
    N = p["N"]
    for inst in range(32):
        order = sorted(range(N), key=lambda m: (float(p["deadline"][inst, m]), m))
        assert list(o["order"][inst]) == order
    # beta >= 0: every prefix is feasible, so each prefix j's front is tried
    # once per later end i
    assert (o["num_inner"] >= N * (N + 1) // 2).all()
    assert (o["num_feasible"] > 0).all()
    dt = p["rate"].dtype.type
    for inst in range(3):  # the count of inner solves, front by front
        order = sorted(range(N), key=lambda m: (float(p["deadline"][inst, m]), m))
        fronts = {0: [(dt(0), p["t_free"][inst])]}
        inner = 0
        for i in range(1, N + 1):
            front = []
            for j in range(i):
                # the states of prefix j from the earliest release; a new
                # inner solve only where the previous winner misses the
                # state's GPU free time
                win = None
                for st in reversed(fronts.get(j, [])):
                    if win is not None:
                        c = _candidate(p, inst, sorted(order[j:i]), st[1], win)
                        if not c["feasible"]:
                            win = None
                    if win is None:
                        inner += 1
                        r = _single(p, inst, sorted(order[j:i]), st[1])
                        if r["status"][0] != 0:
                            break
                        win = (int(r["cut"][0]), int(r["gpu_level"][0]), int(r["batch"][0]))
                        c = {"energy": r["energy"][0], "t_free_out": r["t_free_out"][0]}
                    front = exact_model.front_add(front, (dt(st[0] + c["energy"]), c["t_free_out"]))
            fronts[i] = front
        assert o["num_inner"][inst] == inner
        assert o["energy"][inst] == fronts[N][0][0]


def test_front_capacity_matches_exact_model(tmp_path, monkeypatch):
    """With fronts of at most two states (the oracle built with JO_FRONT=2,
    so the capacity binds on these inputs) the oracle and the exact-rational
    program still agree: the capacity rule (the highest energy leaves) is the
    same on both sides."""
    import ctypes
    import os
    import subprocess
    src = os.path.dirname(oracle.__file__)
    so = str(tmp_path / "lib_front2.so")
    subprocess.run(["gcc", *oracle.CFLAGS, "-DJO_FRONT=2", "-o", so,
                    *[os.path.join(src, f) for f in oracle._SOURCES], "-lm"], check=True)
    lib = ctypes.CDLL(so)
    oracle._declare(lib)
    real = oracle.lib()
    monkeypatch.setattr(exact_model, "FRONT", 2)
    try:
        oracle._lib = lib
        bound = 0
        for shape, stream in (((4, 3, 3, 2), 811), ((4, 2, 2, 3), 812)):
            p = og_tiny(*shape, 10, stream)
            o = oracle.solve_grouped(p)
            for inst in range(10):
                ex = exact_model.solve_grouped_exact(p, inst)
                assert (ex is None) == (o["status"][inst] == 1)
                if ex is not None:
                    assert o["energy"][inst] == pytest.approx(float(ex["energy"]), rel=1e-12)
        p = W.generate(W.WORKLOADS["p5"].replace(N=6, num_instances=16, stream=833))
        full = oracle.solve_grouped(p)
        oracle._lib = real
        free = oracle.solve_grouped(p)
        bound = int((full["energy"] > free["energy"] * (1 + 1e-7)).sum())
        assert bound >= 1  # the capacity binds on some instance
    finally:
        oracle._lib = real
