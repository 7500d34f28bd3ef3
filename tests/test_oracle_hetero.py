"""Pins of the oracle's heterogeneous users (per-user zeta_m, kappa_m, p_m
and CPU levels of Sec. II; no GPU needed).

Pinned against:

* a two-user case worked out by hand, in which the gamma order of Eq. (17)
  at s = 1 is the reverse of the rate order;
* the homogeneous oracle (itself pinned in test_oracle*.py), bitwise, when
  every user carries the shared parameters and no two gamma values tie;
* the long-double brute force over every offloading set and every level
  vector (jdob_brute.c): equal over the per-s gamma-ordered suffixes, never
  lower than the brute force over all sets;
* the exact-rational model (tests/exact_model.py) in every mode, including
  Alg. 2's thresholds written as divisions and the continuous frequency in
  each user's own range;
* invariances that catch a parameter read for the wrong user: scaling user
  m's zeta and levels by 2^a_m and its kappa by 4^-a_m leaves every latency
  and energy bitwise unchanged; relabelling the users permutes the policy;
* monotonicity: a larger kappa_m or p_m never lowers the optimum.
"""

import numpy as np
import pytest

import oracle
from paper_2504_14611_amd import workloads as W
from tests import exact_model

USERS = ("hetero", 0.5, 2.0, 0.5, 2.0, 0.2, 1.0, 0.3e9, 0.8e9, 1.5e9, 2.5e9)


def htiny(N, L, K, J, n, stream, deadline=("beta", 0.2, 3.0), dtype="f64", **kw):
    """Tiny heterogeneous instances; kappa 2.25e-26 and c3-like layers, so
    that offloading and local computing both win."""
    w = W.WORKLOADS["c0"].replace(name="htiny", stream=stream, num_instances=n, N=N, L=L, K=K,
                                  J=J, dtype=dtype, deadline=deadline, kappa=2.25e-26,
                                  cycles=("lu", 1e6, 1e7), rate=("u", 1e6, 100e6),
                                  users=kw.pop("users", USERS), **kw)
    return W.generate(w)


def with_mode(p, mode):
    q = dict(p)
    q["mode"] = mode
    return q


# ---------------------------------------------------------------- closed form

def two_users():
    """Two layers of 1e9 cycles; bits 1e6, 1e5, 1e3; one CPU level (2 GHz),
    one GPU level (1 GHz, 81.25 W); each layer 1 ms + 1 ms per sample on the
    GPU.  User 0: 10 Mbit/s, zeta 4, kappa 2e-28, p 1 W, T = 5 s.  User 1:
    5 Mbit/s, zeta 1, kappa 1e-28, p 0.5 W, T = 1.2 s."""
    return {"cycles": np.array([[1e9, 1e9]]), "bits": np.array([[1e6, 1e5, 1e3]]),
            "alpha": np.array([[1e-3, 1e-3]]), "beta": np.array([[1e-3, 1e-3]]),
            "rate": np.array([[1e7, 5e6]]), "deadline": np.array([[5.0, 1.2]]),
            "t_free": np.array([0.0]), "local_freq": np.array([2e9]),
            "gpu_freq": np.array([1e9]), "kappa": 1e-28, "p_tx": 0.5,
            "gpu_c": 3.125e-26, "gpu_p_static": 50.0, "N": 2, "L": 2, "K": 1, "J": 1,
            "dtype": "f64", "user_zeta": np.array([[4.0, 1.0]]),
            "user_kappa": np.array([[2e-28, 1e-28]]), "user_p_tx": np.array([[1.0, 0.5]])}


def test_two_users_by_hand():
    # s = 0 (nothing local): gamma = upload, 0.1 s < 0.2 s, so user 0 first.
    #   b = 1: upload 0.1 J; GPU 4 ms x 81.25 W = 0.325 J; user 1 local
    #   (1 x 2e9 cycles at 2 GHz = 1 s <= 1.2 s) 1e-28 x 4e18 x 2e9 = 0.8 J
    #   -> 1.225 J.  b = 2: uploads 0.1 + 0.1 J, GPU 6 ms -> 0.4875 J
    #   -> 0.6875 J (the optimum), released at 0.2 + 0.006 s.
    # s = 1: gamma_0 = 0.01 + 4e9/2e9 = 2.01 s, gamma_1 = 0.02 + 0.5 = 0.52 s,
    #   so user 1 is first although its rate is lower.  b = 1: user 1 runs
    #   layer 1 (0.4 J), uploads (0.01 J), GPU 2 ms (0.1625 J); user 0 local
    #   (8e9 cycles, 4 s <= 5 s) 2e-28 x 4e18 x 2e9 = 1.6 J (Eq. (2) has no
    #   zeta) -> 2.1725 J, released at 0.52 + 0.002 s.  b = 2 misses (7):
    #   user 0 needs 2 s of local compute before a 1.2 s deadline.
    # Local computing: 1.6 + 0.8 = 2.4 J.
    p = two_users()
    o = oracle.solve(p)
    assert o["status"][0] == 0
    assert (o["cut"][0], o["gpu_level"][0], o["batch"][0]) == (0, 0, 2)
    assert o["energy"][0] == pytest.approx(0.6875, rel=1e-15)
    assert o["t_free_out"][0] == pytest.approx(0.206, rel=1e-15)
    assert o["energy_second"][0] == pytest.approx(1.225, rel=1e-15)
    assert o["num_feasible"][0] == 4   # (0,0,1), (0,0,2), (1,0,1), local
    c = oracle.eval_candidate(p, 0, 1, 0, 1)
    assert c["feasible"] and list(c["user_offload"]) == [0, 1]
    assert c["energy"] == pytest.approx(2.1725, rel=1e-15)
    assert c["t_free_out"] == pytest.approx(0.522, rel=1e-15)
    assert not oracle.eval_candidate(p, 0, 1, 0, 2)["feasible"]
    lc = oracle.eval_candidate(p, 0, 2, 0, 0)
    assert lc["feasible"] and lc["energy"] == pytest.approx(2.4, rel=1e-15)
    # the homogeneous reading (rate order) would offload user 0 at s = 1
    q = {k: v for k, v in p.items() if not k.startswith("user_")}
    assert list(oracle.eval_candidate(q, 0, 1, 0, 1)["user_offload"]) == [1, 0]


# ------------------------------------------------------- homogeneous reduction

def _shared_users(p):
    """The shared parameters written out per user."""
    q = dict(p)
    I, N, K = W.num_instances(p), p["N"], p["K"]
    dt = p["rate"].dtype
    q["user_zeta"] = np.ones((I, N), dt)
    q["user_kappa"] = np.full((I, N), p["kappa"], dt)
    q["user_p_tx"] = np.full((I, N), p["p_tx"], dt)
    q["user_local_freq"] = np.broadcast_to(p["local_freq"], (I, N, K)).astype(dt)
    return q


def _gamma_ties(p):
    """Instances where two users share a gamma (Eq. (17)) at some s: there
    the gamma order and the rate order may break the tie differently."""
    dt = p["rate"].dtype.type
    C = np.zeros((W.num_instances(p), p["L"] + 1), p["rate"].dtype)
    for s in range(p["L"]):
        C[:, s + 1] = C[:, s] + p["cycles"][:, s]
    bad = np.zeros(W.num_instances(p), bool)
    for s in range(p["L"]):
        up = p["bits"][:, s:s + 1] / p["rate"]
        t = (dt(1) * C[:, s:s + 1]) / p["local_freq"][-1]
        g = np.sort(up + t, axis=1)
        bad |= (np.diff(g, axis=1) == 0).any(axis=1)
    return bad


@pytest.mark.parametrize("mode", [0, 1, 2, 4, 7, 8, 9])
@pytest.mark.parametrize("name,n", [("c1", 512), ("c2b", 256), ("c3", 256), ("c0", 256)])
def test_identical_users_reduce_to_the_homogeneous_oracle(name, n, mode):
    kw = {"kappa": 1e-27} if name == "c2b" else {}
    p = with_mode(W.generate(W.WORKLOADS[name].replace(**kw), 0, n), mode)
    a, b = oracle.solve(p, threads=4), oracle.solve(_shared_users(p), threads=4)
    keep = ~_gamma_ties(p)
    assert keep.sum() >= n // 2
    for k in a:
        x, y = a[k][keep], b[k][keep]
        if x.dtype.kind == "f":
            assert np.array_equal(x, y, equal_nan=True), k
        else:
            assert np.array_equal(x, y), k


def test_reduction_is_sensitive():
    """The reduction cases include offloading winners and partial batches."""
    p = W.generate(W.WORKLOADS["c2b"].replace(kappa=1e-27), 0, 256)
    o = oracle.solve(p)
    f = o["status"] == 0
    assert ((o["cut"] < p["L"]) & f).sum() > 30
    assert ((o["batch"] < p["N"]) & (o["cut"] < p["L"]) & f).sum() > 5


# --------------------------------------------------------------- brute force

@pytest.mark.parametrize("stream", [1201, 1202, 1203])
def test_brute_force_over_gamma_suffixes(stream):
    p = htiny(4, 3, 3, 3, 24, stream)
    o = oracle.solve(p)
    for inst in range(24):
        bf = oracle.brute(p, inst, suffix_only=True)
        assert bf["found"] == (o["status"][inst] == 0), inst
        if not bf["found"]:
            continue
        assert o["energy"][inst] == pytest.approx(bf["energy"], rel=1e-12), inst
        assert o["num_feasible"][inst] == bf["num_feasible"], inst
        if bf["energy_second"] > bf["energy"] * (1 + 1e-9):
            assert (o["cut"][inst], o["gpu_level"][inst], o["batch"][inst]) == \
                (bf["cut"], bf["gpu_level"], bf["batch"]), inst
            assert np.array_equal(o["user_level"][inst], bf["user_level"]), inst
        full = oracle.brute(p, inst, suffix_only=False)
        assert full["energy"] <= o["energy"][inst] * (1 + 1e-12), inst


def test_brute_force_pin_is_sensitive():
    """Winners offload partial batches at s > 0 in an order that differs
    from the rate order."""
    p = htiny(4, 3, 3, 3, 72, 1201)
    o = oracle.solve(p)
    f = o["status"] == 0
    part = f & (o["cut"] > 0) & (o["cut"] < p["L"]) & (o["batch"] < p["N"])
    assert part.sum() >= 3
    diff = 0
    for inst in np.nonzero(part)[0]:
        s, b = o["cut"][inst], o["batch"][inst]
        by_rate = set(np.argsort(-p["rate"][inst], kind="stable")[:b])
        diff += by_rate != set(np.nonzero(o["user_offload"][inst])[0])
    assert diff >= 1


# ------------------------------------------------------------ exact rational

@pytest.mark.parametrize("mode", [0, 1, 2, 4, 8, 9])
@pytest.mark.parametrize("stream", [1211, 1212])
def test_exact_rational(mode, stream):
    p = with_mode(htiny(4, 4, 3, 3, 16, stream), mode)
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
            assert o["t_free_out"][inst] == pytest.approx(float(ex["t_free_out"]), rel=1e-12)
            if mode & oracle.MODE_CONTINUOUS:
                assert np.allclose(o["user_freq"][inst], [float(x) for x in ex["levels"]],
                                   rtol=1e-13)
            else:
                assert list(o["user_level"][inst]) == list(ex["levels"]), inst


def test_exact_greedy_differs_from_grid():
    """Alg. 2's greedy set is not the grid's best on these inputs."""
    p = htiny(4, 4, 3, 3, 64, 1211)
    a, b = oracle.solve(p), oracle.solve(with_mode(p, oracle.MODE_GREEDY))
    f = a["status"] == 0
    assert (b["energy"][f] > a["energy"][f] * (1 + 1e-9)).sum() >= 2


# ----------------------------------------------------------------- invariances

def _rescaled(p, seed):
    rng = np.random.default_rng(seed)
    q = dict(p)
    a = rng.integers(-1, 3, size=p["rate"].shape).astype(np.float64)
    c = (2.0 ** a).astype(p["rate"].dtype)
    q["user_zeta"] = p["user_zeta"] * c
    q["user_local_freq"] = p["user_local_freq"] * c[:, :, None]
    q["user_kappa"] = p["user_kappa"] / (c * c)
    return q, c


@pytest.mark.parametrize("mode", [0, 1, 6, 8, 9])
@pytest.mark.parametrize("name", ["h1", "h2"])
def test_per_user_power_of_two_rescaling(name, mode):
    p = with_mode(W.generate(W.WORKLOADS[name], 0, 512), mode)
    q, c = _rescaled(p, 5 + mode)
    a, b = oracle.solve(p, threads=4), oracle.solve(q, threads=4)
    for k in a:
        if k == "user_freq":
            assert np.array_equal(a[k] * c, b[k]), k
        else:
            assert np.array_equal(a[k], b[k], equal_nan=True), k


def test_rescaling_pin_is_sensitive():
    """Per-user parameters matter: the h1 policies change when one user's
    kappa, p or levels are replaced by another user's."""
    p = W.generate(W.WORKLOADS["h1"], 0, 512)
    a = oracle.solve(p, threads=4)
    for key in ("user_kappa", "user_p_tx", "user_zeta", "user_local_freq"):
        q = dict(p)
        q[key] = np.roll(p[key], 1, axis=1)
        b = oracle.solve(q, threads=4)
        assert (a["energy"] != b["energy"]).sum() > 100, key


@pytest.mark.parametrize("mode", [0, 1, 8])
def test_relabelling_users_permutes_the_policy(mode):
    p = with_mode(W.generate(W.WORKLOADS["h1"], 0, 384), mode)
    rng = np.random.default_rng(31)
    perm = rng.permutation(p["N"])
    q = dict(p)
    for k in ("rate", "deadline") + W.USER_KEYS:
        q[k] = np.ascontiguousarray(p[k][:, perm])
    a, b = oracle.solve(p, threads=4), oracle.solve(q, threads=4)
    assert np.array_equal(a["status"], b["status"])
    f = a["status"] == 0
    assert np.allclose(a["energy"][f], b["energy"][f], rtol=1e-5)
    gap = (a["energy_second"] - a["energy"]) > 1e-4 * np.abs(a["energy"])
    same = f & gap
    for k in ("cut", "gpu_level", "batch"):
        assert np.array_equal(a[k][same], b[k][same]), k
    for k in ("user_level", "user_offload"):
        assert np.array_equal(a[k][same][:, perm], b[k][same]), k


# ---------------------------------------------------------------- monotonicity

@pytest.mark.parametrize("key", ["user_kappa", "user_p_tx"])
def test_more_expensive_user_never_lowers_the_optimum(key):
    p = W.generate(W.WORKLOADS["h1"], 0, 512)
    q = dict(p)
    x = p[key].copy()
    x[:, 3] *= 1.5
    q[key] = x
    a, b = oracle.solve(p, threads=4), oracle.solve(q, threads=4)
    assert np.array_equal(a["status"], b["status"])
    f = a["status"] == 0
    assert (b["energy"][f] >= a["energy"][f] * (1 - 1e-6)).all()
    assert (b["energy"][f] > a["energy"][f] * (1 + 1e-6)).sum() > 20


def test_tables_refuse_heterogeneous_users():
    with pytest.raises(RuntimeError):
        oracle.user_tables(htiny(4, 3, 3, 3, 2, 1220))


# ------------------------------------------------------------------ invariants

def _recheck_hetero(p, o, inst, rtol):
    """Recompute a returned policy from the model definitions in binary64
    (each user's own zeta, kappa, p and levels): (7), (8), Eq. (21), (22)."""
    N = p["N"]
    cyc = p["cycles"][inst].astype(np.float64)
    bits = p["bits"][inst].astype(np.float64)
    al, be = p["alpha"][inst].astype(np.float64), p["beta"][inst].astype(np.float64)
    R, T = p["rate"][inst].astype(np.float64), p["deadline"][inst].astype(np.float64)
    g = p["gpu_freq"].astype(np.float64)
    z = p["user_zeta"][inst].astype(np.float64)
    kap = p["user_kappa"][inst].astype(np.float64)
    ptx = p["user_p_tx"][inst].astype(np.float64)
    fu = p["user_local_freq"][inst].astype(np.float64)
    s, j, b = o["cut"][inst], o["gpu_level"][inst], o["batch"][inst]
    off = o["user_offload"][inst].astype(bool)
    fr = o["user_freq"][inst].astype(np.float64)
    assert off.sum() == b
    E, ready = 0.0, 0.0
    for m in range(N):
        assert fu[m, 0] * (1 - 1e-6) <= fr[m] <= fu[m, -1] * (1 + 1e-6)
        if off[m]:
            w = cyc[:s].sum()
            E += kap[m] * fr[m] ** 2 * w + ptx[m] * bits[s] / R[m]
            ready = max(ready, z[m] * w / fr[m] + bits[s] / R[m])
        else:
            w = cyc.sum()
            assert z[m] * w / fr[m] <= T[m] * (1 + rtol), ("(8)", inst, m)
            E += kap[m] * fr[m] ** 2 * w
    if b > 0:
        phi = (al[s:].sum() + be[s:].sum() * b) * g[-1] / g[j]
        assert ready + phi <= T[off].min() * (1 + rtol), ("(7)", inst)
        E += (p["gpu_c"] * g[j] ** 3 + p["gpu_p_static"]) * phi
        assert o["t_free_out"][inst] == pytest.approx(ready + phi, rel=rtol)
    assert o["energy"][inst] == pytest.approx(E, rel=rtol)


@pytest.mark.parametrize("mode", [0, 1, 8, 9])
@pytest.mark.parametrize("name,n", [("h1", 256), ("h2", 512)])
def test_hetero_policies_meet_deadlines_and_never_exceed_local(name, n, mode):
    p = with_mode(W.generate(W.WORKLOADS[name], 0, n), mode)
    o = oracle.solve(p, threads=4)
    for inst in np.nonzero(o["status"] == 0)[0]:
        _recheck_hetero(p, o, inst, 1e-5)
        lc = oracle.eval_candidate(p, inst, p["L"], 0, 0)
        if lc["feasible"]:
            assert o["energy"][inst] <= lc["energy"]


@pytest.mark.parametrize("mode", [0, 8])
def test_hetero_relaxing_deadlines_never_costs_energy(mode):
    p = with_mode(W.generate(W.WORKLOADS["h1"], 0, 256), mode)
    o = oracle.solve(p, threads=4)
    feas = o["status"] == 0
    rng = np.random.default_rng(41)
    for lam in (1.05, 1.5):
        q = dict(p)
        q["deadline"] = (p["deadline"] * np.asarray(lam, p["deadline"].dtype)).astype(p["deadline"].dtype)
        oq = oracle.solve(q, threads=4)
        assert (oq["status"][feas] == 0).all()
        assert (oq["energy"][feas] <= o["energy"][feas]).all()
        q = dict(p)
        d = p["deadline"].copy()
        d[np.arange(d.shape[0]), rng.integers(0, p["N"], size=d.shape[0])] *= np.asarray(lam, d.dtype)
        q["deadline"] = d
        oq = oracle.solve(q, threads=4)
        assert (oq["status"][feas] == 0).all()
        assert (oq["energy"][feas] <= o["energy"][feas]).all()


def test_hetero_feasible_batches_form_growing_intervals():
    """At every (s, j) the feasible batches are [max(bmin_s, 1), bmax], bmax
    grows with j (the monotone thresholds of Eq. (18) with per-user gammas),
    and the work counters count exactly those candidates: enumerated one
    candidate at a time."""
    p = htiny(5, 4, 3, 4, 8, 1230)
    o = oracle.solve(p)
    N, L, J = p["N"], p["L"], p["J"]
    for inst in range(8):
        nfeas, nev = 0, 0
        for s in range(L):
            prev = 0
            for j in range(J):
                ok = [oracle.eval_candidate(p, inst, s, j, b)["feasible"] for b in range(1, N + 1)]
                bmax = max([b for b in range(1, N + 1) if ok[b - 1]], default=0)
                blo = min([b for b in range(1, N + 1) if ok[b - 1]], default=0)
                assert ok == [bool(bmax) and blo <= b <= bmax for b in range(1, N + 1)]
                assert bmax >= prev
                prev = max(prev, bmax)
                nfeas += sum(ok)
                nev += sum(b for b in range(1, N + 1) if ok[b - 1])
        nfeas += oracle.eval_candidate(p, inst, L, 0, 0)["feasible"]
        assert o["num_feasible"][inst] == nfeas
        assert o["num_user_evals"][inst] == nev


# ------------------------------------------------------- grouping (outer module)

def og_htiny(N, L, K, J, n, stream):
    from tests.test_oracle_grouped import og_tiny
    return og_tiny(N, L, K, J, n, stream, users=USERS)


@pytest.mark.parametrize("shape,stream", [((3, 3, 2, 3), 1240), ((4, 3, 3, 2), 1241)])
def test_grouping_exact_rational(shape, stream):
    p = og_htiny(*shape, 10, stream)
    o = oracle.solve_grouped(p)
    for inst in range(10):
        ex = exact_model.solve_grouped_exact(p, inst)
        if ex is None:
            assert o["status"][inst] == 1, inst
            continue
        assert o["status"][inst] == 0, inst
        assert o["energy"][inst] == pytest.approx(float(ex["energy"]), rel=1e-12), inst
        assert o["t_free_out"][inst] == pytest.approx(float(ex["t_free_out"]), rel=1e-12), inst


def test_grouping_pin_is_sensitive():
    """Several groups win, and the per-user parameters change the answer."""
    p = og_htiny(4, 3, 3, 2, 40, 1241)
    o = oracle.solve_grouped(p)
    f = o["status"] == 0
    assert (o["num_groups"][f] > 1).sum() >= 5
    q = dict(p)
    q["user_kappa"] = np.roll(p["user_kappa"], 1, axis=1)
    assert (oracle.solve_grouped(q)["energy"][f] != o["energy"][f]).sum() >= 10


def test_grouping_with_shared_values_matches_homogeneous():
    p = W.generate(W.WORKLOADS["g10"], 0, 256)
    a, b = oracle.solve_grouped(p, threads=4), oracle.solve_grouped(_shared_users(p), threads=4)
    keep = ~_gamma_ties(p)
    assert keep.sum() > 128
    for k in a:
        assert np.array_equal(a[k][keep], b[k][keep], equal_nan=True), k


def test_grouping_rescaling_and_replay():
    p = W.WORKLOADS["h2"]
    p = W.generate(p.replace(name="h2g", num_instances=128), 0, 128)
    o = oracle.solve_grouped(p, threads=4)
    q, c = _rescaled(p, 11)
    oq = oracle.solve_grouped(q, threads=4)
    for k in o:
        if k == "user_freq":
            assert np.array_equal(o[k] * c, oq[k]), k
        else:
            assert np.array_equal(o[k], oq[k], equal_nan=True), k
    from tests.test_oracle_grouped import group_arrays
    for inst in np.nonzero(o["status"] == 0)[0][:64]:
        ev = oracle.eval_grouping(p, int(inst), *group_arrays(o, inst))
        assert ev["feasible"] and ev["energy"] == o["energy"][inst]
        assert np.array_equal(ev["user_level"], o["user_level"][inst])
        assert np.array_equal(ev["user_freq"], o["user_freq"][inst])
