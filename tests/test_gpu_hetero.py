"""GPU parity of heterogeneous users (per-user zeta, kappa, transmit power
and CPU levels; jdob_solve_batch with the jdob_problem.user_* arrays)
through the C ABI, against the oracle on the same inputs.

Covers the workloads h1 (8 levels per user) and h2 (Table I, continuous) in
every search mode, shapes at the kernel's limits (1 and 64 users, 1 and 64
levels, GPU levels beyond one wave), inputs with only some per-user arrays,
zero-work layers, tied gammas and a busy GPU, the shared parameters written
per user against the homogeneous kernel, and the full h1 and h2 batches,
every instance;
then the outer grouping with heterogeneous users (jdob_solve_grouped).
Comparison rules: tests/parity.py, compare_grouped in tests/test_gpu_grouped.py.  Every case prints its name, shape, mode
and entry point before touching the GPU.
"""

import numpy as np
import pytest

import oracle
from paper_2504_14611_amd import jdob
from paper_2504_14611_amd import workloads as W
from tests.parity import compare
from tests.test_gpu_parity import THREADS, _edge, _say

pytestmark = pytest.mark.gpu


def with_mode(p, mode):
    q = dict(p)
    q["mode"] = mode
    return q


def check(prob, label, freq=True):
    import torch
    _say(f"{label} mode={prob.get('mode', 0)} users={[k for k in W.USER_KEYS if prob.get(k) is not None]}",
         prob)
    d = jdob.to_device(prob)
    gpu = jdob.to_host(jdob.solve_batch(d, freq=freq))
    torch.cuda.synchronize()
    ora = oracle.solve(prob, threads=THREADS)
    st = compare(prob, gpu, ora, label=label)
    print(f"[gpu] {label}: ok {st}", flush=True)
    return gpu, ora


@pytest.mark.parametrize("mode", [0, 1, 2, 4, 7, 8, 9])
@pytest.mark.parametrize("name,n", [("h1", 4096), ("h2", 4096)])
def test_hetero_prefix(name, n, mode):
    check(with_mode(W.generate(W.WORKLOADS[name], 0, n), mode), f"{name}[:{n}]")


def test_hetero_cases_are_not_homogeneous():
    """The orders differ from the rate order and partial batches win."""
    p = W.generate(W.WORKLOADS["h1"], 0, 2048)
    o = oracle.solve(p, threads=THREADS)
    f = (o["status"] == 0) & (o["cut"] < p["L"])
    assert (f & (o["batch"] < p["N"])).sum() > 300
    diff = 0
    for inst in np.nonzero(f)[0][:400]:
        b = o["batch"][inst]
        by_rate = set(np.argsort(-p["rate"][inst], kind="stable")[:b])
        diff += by_rate != set(np.nonzero(o["user_offload"][inst])[0])
    assert diff > 50


HETERO_EDGES = {
    "N1": ("h1", 512, dict(N=1), (0, 1, 8)),
    "N2": ("h1", 512, dict(N=2), (0, 1)),
    "N64": ("h1", 24, dict(N=64, L=6, J=8), (0, 1, 8)),
    "K1": ("h1", 512, dict(K=1), (0, 1, 8)),
    "K2": ("h1", 512, dict(K=2), (0, 9)),
    "K5": ("h1", 256, dict(K=5), (0, 1)),
    "K64": ("h1", 64, dict(K=64, N=8, L=8), (0, 1)),
    "J1": ("h1", 512, dict(J=1), (0, 1)),
    "J100": ("h1", 128, dict(J=100, N=8), (0, 1, 3)),
    "J256": ("h2", 64, dict(J=256), (8, 9)),
    "L1": ("h1", 512, dict(L=1), (0, 4)),
    "f64_h1": ("h1", 512, dict(dtype="f64"), (0, 1, 8)),
    "f64_h2": ("h2", 512, dict(dtype="f64"), (8, 9)),
    # the rows' runs of partition points: four per run up to 16 users (with
    # a short last run), two up to 32, one beyond
    "N16_L5": ("h1", 256, dict(N=16, L=5), (0, 1, 8)),
    "N24_L7": ("h1", 256, dict(N=24, L=7), (0, 1, 8)),
    "N40_L5": ("h1", 64, dict(N=40, L=5, J=8), (0, 1, 8)),
    "I1": ("h1", 1, {}, (0,)),
    "I1001": ("h1", 1001, {}, (0, 1)),
}


@pytest.mark.parametrize("case", sorted(HETERO_EDGES))
def test_hetero_edge_shapes(case):
    base, n, kw, modes = HETERO_EDGES[case]
    prob = _edge(base, n, 1300 + sorted(HETERO_EDGES).index(case), **kw)
    for mode in modes:
        check(with_mode(prob, mode), f"{case} mode={mode}")


@pytest.mark.parametrize("keep", [("user_zeta",), ("user_kappa",), ("user_p_tx",),
                                  ("user_local_freq",), ("user_zeta", "user_local_freq")])
def test_some_per_user_arrays(keep):
    p = W.generate(W.WORKLOADS["h1"], 0, 1024)
    for k in W.USER_KEYS:
        if k not in keep:
            p[k] = None
    check(p, f"h1 only {'+'.join(keep)}")
    check(with_mode(p, 9), f"h1 only {'+'.join(keep)} greedy+continuous")


def test_hetero_zeros_ties_and_busy_gpu():
    p = W.generate(W.WORKLOADS["h1"], 0, 2048)
    p["cycles"][:512, :3] = 0                      # C[s] = 0 for s <= 3
    p["bits"][256:768, 5] = 0                      # nothing to upload after layer 5
    for k in ("rate", "deadline") + W.USER_KEYS:   # users 0 and 1 identical: tied gamma
        p[k][1024:, 1] = p[k][1024:, 0]
    rng = np.random.default_rng(23)
    p["t_free"] = rng.uniform(0, 0.02, size=2048).astype(np.float32)
    for mode in (0, 1, 8):
        check(with_mode(p, mode), f"zeros+ties+t_free mode={mode}")


def test_shared_values_match_the_homogeneous_kernel():
    """The heterogeneous kernel with every user carrying the shared values
    equals the homogeneous kernel wherever no two gammas tie (where they
    tie, the gamma order and the rate order may differ)."""
    import torch
    from tests.test_oracle_hetero import _gamma_ties, _shared_users
    for name, n, mode in (("c3", 4096, 0), ("c2b", 2048, 1), ("c1", 2048, 8)):
        p = with_mode(W.generate(W.WORKLOADS[name], 0, n), mode)
        q = _shared_users(p)
        _say(f"{name} shared values per user, mode={mode}", q, "jdob_solve_batch (both paths)")
        a = jdob.to_host(jdob.solve_batch(jdob.to_device(p), freq=True))
        b = jdob.to_host(jdob.solve_batch(jdob.to_device(q), freq=True))
        torch.cuda.synchronize()
        keep = ~_gamma_ties(p)
        assert keep.sum() > n // 2
        for k in a:
            assert np.array_equal(a[k][keep], b[k][keep], equal_nan=True), (name, k)


@pytest.mark.parametrize("name", ["h1", "h2"])
def test_hetero_full_size_every_instance(name):
    """The whole batch (h1: 262,144 instances, 16 users with 8 levels each;
    h2: Table I, continuous) in the benchmark's launch configuration, every
    instance compared with the oracle (about 3 s on 16 threads)."""
    import torch
    w = W.WORKLOADS[name]
    prob = W.generate(w)
    _say(f"{name} full", prob)
    gpu = jdob.to_host(jdob.solve_batch(jdob.to_device(prob), counters=False))
    torch.cuda.synchronize()
    ora = oracle.solve(prob, threads=THREADS)
    st = compare(prob, gpu, ora, label=f"{name} full")
    print(f"[gpu] {name} full: ok {st}", flush=True)


# ------------------------------------------------------- grouping (outer module)

def check_grouped(prob, label):
    from tests.test_gpu_grouped import check as grouped_check
    return grouped_check(prob, f"{label} users={[k for k in W.USER_KEYS if prob.get(k) is not None]}",
                         freq=True)


@pytest.mark.parametrize("name,n,mode", [("h2", 1024, 8), ("h2", 512, 9), ("h2", 256, 0),
                                         ("h1", 256, 0), ("h1", 128, 1), ("h1", 128, 8)])
def test_hetero_grouped(name, n, mode):
    w = W.WORKLOADS[name]
    if name == "h1":   # 10 users, deadlines spread as in the grouping workloads
        w = w.replace(N=10, deadline=("beta", 0.0, 10.0))
    p = with_mode(W.generate(w.replace(num_instances=n)), mode)
    check_grouped(p, f"{name}[:{n}] grouped mode={mode}")


@pytest.mark.parametrize("case,kw", [("N1", dict(N=1)), ("N2", dict(N=2)),
                                     ("N64", dict(N=64, L=4, J=4)), ("f64", dict(dtype="f64")),
                                     ("K1", dict(K=1))])
def test_hetero_grouped_edges(case, kw):
    n = 8 if case == "N64" else 128
    p = _edge("h2", n, 1400 + len(case), **kw)
    check_grouped(p, f"grouped {case}")


def test_hetero_grouped_some_arrays_and_busy_gpu():
    p = W.generate(W.WORKLOADS["h2"].replace(num_instances=256))
    p["user_zeta"] = None
    p["user_p_tx"] = None
    p["t_free"] = np.random.default_rng(5).uniform(0, 0.002, size=256).astype(np.float32)
    check_grouped(p, "h2 grouped kappa+levels only, busy GPU")


def test_hetero_grouped_shared_values_match_homogeneous_grouping():
    import torch
    from tests.test_oracle_hetero import _gamma_ties, _shared_users
    p = W.generate(W.WORKLOADS["g10"], 0, 512)
    q = _shared_users(p)
    _say("g10 shared values per user", q, "jdob_solve_grouped (both paths)")
    a = jdob.to_host(jdob.solve_grouped(jdob.to_device(p), freq=True))
    b = jdob.to_host(jdob.solve_grouped(jdob.to_device(q), freq=True))
    torch.cuda.synchronize()
    keep = ~_gamma_ties(p)
    assert keep.sum() > 256
    for k in a:
        assert np.array_equal(a[k][keep], b[k][keep], equal_nan=True), k
