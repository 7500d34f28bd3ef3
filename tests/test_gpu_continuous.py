"""GPU parity of the continuous CPU frequency (JDOB_MODE_CONTINUOUS_CPU: Eq.
(20) with its clamp) through the C ABI, against the oracle in the same mode.

Covers the paper-parameter workloads (Table I: p4a, p4b, p5), the synthetic
workloads with the continuous bit alone and with every other mode bit,
the shapes at the kernel's chunk boundaries, both stages against the fused
entry point, the outer grouping, and the full p4a and p4b batches, every
instance.
Comparison rules: tests/parity.py (single solves), compare_grouped in
tests/test_gpu_grouped.py (grouping); both compare the returned CPU
frequencies bitwise where the decisions agree.  Every case prints its name,
shape, mode and entry point before touching the GPU.
"""

import numpy as np
import pytest

import oracle
from paper_2504_14611_amd import jdob
from paper_2504_14611_amd import workloads as W
from tests.parity import compare
from tests.test_gpu_grouped import check as check_grouped
from tests.test_gpu_parity import THREADS, _edge, _say

pytestmark = pytest.mark.gpu

CONT = jdob.JDOB_MODE_CONTINUOUS_CPU


def with_mode(p, mode):
    q = dict(p)
    q["mode"] = mode
    return q


def check(prob, label, freq=None):
    import torch
    _say(f"{label} mode={prob.get('mode', 0)}", prob)
    d = jdob.to_device(prob)
    gpu = jdob.to_host(jdob.solve_batch(d, freq=freq))
    torch.cuda.synchronize()
    ora = oracle.solve(prob, threads=THREADS)
    st = compare(prob, gpu, ora, label=label)
    print(f"[gpu] {label}: ok {st}", flush=True)
    return gpu, ora


def test_user_freq_is_allocated_for_continuous_problems():
    p = W.generate(W.WORKLOADS["p4a"], 0, 4)
    assert jdob.alloc_policy(jdob.to_device(p))["user_freq"] is not None
    assert jdob.alloc_policy(jdob.to_device(with_mode(p, 0)))["user_freq"] is None


@pytest.mark.parametrize("name,n", [("p4a", 8192), ("p4b", 8192), ("p5", 8192)])
def test_paper_parameter_prefix(name, n):
    p = W.generate(W.WORKLOADS[name], 0, n)
    assert p["mode"] == CONT
    gpu, ora = check(p, f"{name}[:{n}]")
    f = ora["status"] == 0
    assert f.sum() > n // 2


def _kappa(prob, kappa):
    prob["kappa"] = kappa
    return prob


PREFIXES = {
    "c1": lambda: W.generate(W.WORKLOADS["c1"], 0, 1024),
    "c2b_k27": lambda: _kappa(W.generate(W.WORKLOADS["c2b"], 0, 2048), 1e-27),
    "c3": lambda: W.generate(W.WORKLOADS["c3"], 0, 2048),
    "c4b": lambda: W.generate(W.WORKLOADS["c4b"], 0, 48),
    "p4a": lambda: W.generate(W.WORKLOADS["p4a"], 0, 4096),
}


@pytest.mark.parametrize("extra", [0, 1, 2, 3, 4, 7])
@pytest.mark.parametrize("name", sorted(PREFIXES))
def test_continuous_with_every_mode(name, extra):
    check(with_mode(PREFIXES[name](), CONT | extra), f"{name} cont|{extra}")


def test_continuous_picks_frequencies_between_the_levels():
    """The parity cases above are not the discrete ones in disguise: many
    users run strictly between f_0 and f_{K-1}."""
    p = with_mode(PREFIXES["c2b_k27"](), CONT)
    o = oracle.solve(p, threads=THREADS)
    f = o["status"] == 0
    lo, hi = p["local_freq"][0], p["local_freq"][-1]
    inside = (o["user_freq"][f] > lo) & (o["user_freq"][f] < hi)
    assert inside.sum() > 1000


@pytest.mark.parametrize("mode", [0, 1, 7])
def test_discrete_modes_return_the_level_frequencies(mode):
    """user_freq requested in a discrete mode: the frequency of each user's
    level, bitwise the oracle's."""
    p = with_mode(W.generate(W.WORKLOADS["c1"], 0, 1024), mode)
    gpu, _ = check(p, f"c1 discrete freq mode={mode}", freq=True)
    f = gpu["status"] == 0
    lv = gpu["user_level"][f].astype(np.int64)
    assert np.array_equal(gpu["user_freq"][f], p["local_freq"][lv])


CONT_EDGES = {
    "N1": ("c1", 512, dict(N=1), (0, 1)),
    "N65": ("c4b", 48, dict(N=65, L=12, K=8, J=16), (0, 1)),
    "N129": ("c4b", 32, dict(N=129, L=10, K=8, J=16), (0, 1)),
    "N1024": ("c4b", 3, dict(N=1024, L=3, K=4, J=4), (0, 1)),
    # f_0 == f_{K-1}: every frequency is the one level
    "K1": ("c1", 512, dict(K=1, local_f=(2.0e9, 2.0e9)), (0, 1)),
    "K2": ("c1", 512, dict(K=2), (0, 1, 7)),
    "J1": ("c1", 512, dict(J=1), (0, 1)),
    "L1": ("c1", 512, dict(L=1), (0, 4)),
    "J100": ("c2b", 256, dict(J=100), (0, 1, 3)),
    "J256": ("c1", 64, dict(J=256, N=8, L=6), (0, 1)),
    "f64_c1": ("c1", 1024, dict(dtype="f64"), (0, 1, 7)),
    "f64_p4a": ("p4a", 1024, dict(dtype="f64"), (0, 1)),
    "f64_N70": ("c4b", 16, dict(N=70, L=8, K=8, J=8, dtype="f64"), (0, 1)),
    "I1": ("c3", 1, {}, (0,)),
    "I1001": ("c3", 1001, {}, (0, 1)),
}


@pytest.mark.parametrize("case", sorted(CONT_EDGES))
def test_continuous_edge_shapes(case):
    base, n, kw, extras = CONT_EDGES[case]
    prob = _edge(base, n, 1100 + sorted(CONT_EDGES).index(case), **kw)
    for extra in extras:
        check(with_mode(prob, CONT | extra), f"{case} cont|{extra}")


def test_continuous_zero_cycles_ties_and_busy_gpu():
    """Layers without cycles (C[s] = 0 before the first costly layer: f_0,
    no CPU energy), tied rates and a GPU busy at the start."""
    p = _kappa(W.generate(W.WORKLOADS["c2b"], 0, 2048), 1e-27)
    p["rate"][:, 1] = p["rate"][:, 0]
    p["rate"][:, 5:9] = p["rate"][:, 4:5]
    p["cycles"][:512, ::3] = 0
    p["cycles"][512:768, :4] = 0
    p["bits"][256:1024, 4] = 0
    rng = np.random.default_rng(19)
    p["t_free"] = rng.uniform(0, 0.05, size=2048).astype(np.float32)
    for extra in (0, 1, 5):
        check(with_mode(p, CONT | extra), f"zeros+ties+t_free cont|{extra}")


def test_continuous_stage_parity():
    """eval_joint(eval_user_tables(x)) == solve_batch(x) bitwise with a
    continuous CPU frequency."""
    import torch
    for name, n in (("p4a", 2048), ("c2b", 1024), ("c4b", 32)):
        prob = W.generate(W.WORKLOADS[name], 0, n)
        for extra in (0, 1, 7):
            q = with_mode(prob, CONT | extra)
            _say(f"{name} cont|{extra}", q, "jdob_eval_user_tables + jdob_eval_joint")
            d = jdob.to_device(q)
            fused = jdob.to_host(jdob.solve_batch(d))
            tabs = jdob.eval_user_tables(d)
            joint = jdob.to_host(jdob.eval_joint(d, tabs))
            torch.cuda.synchronize()
            for k in fused:
                assert np.array_equal(fused[k], joint[k], equal_nan=True), (name, extra, k)


@pytest.mark.parametrize("name,n,extra", [("p5", 1024, 0), ("p5", 512, 1), ("g10", 512, 0),
                                          ("g10", 256, 3)])
def test_continuous_grouped(name, n, extra):
    p = with_mode(W.generate(W.WORKLOADS[name], 0, n), CONT | extra)
    check_grouped(p, f"{name}[:{n}] grouped cont|{extra}")


def test_continuous_grouped_f64_and_discrete_freq():
    p = _edge("p5", 256, 1190, dtype="f64")
    check_grouped(p, "p5 f64 grouped")
    q = with_mode(W.generate(W.WORKLOADS["g10"], 0, 256), 0)
    check_grouped(q, "g10 grouped discrete freq", freq=True)


@pytest.mark.parametrize("name", ["p4a", "p4b"])
def test_paper_parameters_full_size_every_instance(name):
    """The whole p4a and p4b batches (Table I, continuous frequency) in the
    benchmark's launch configuration, every instance compared with the
    oracle."""
    import torch
    w = W.WORKLOADS[name]
    prob = W.generate(w)
    _say(f"{name} full", prob)
    d = jdob.to_device(prob)
    gpu = jdob.to_host(jdob.solve_batch(d, counters=False))
    torch.cuda.synchronize()
    ora = oracle.solve(prob, threads=THREADS)
    st = compare(prob, gpu, ora, label=f"{name} full")
    print(f"[gpu] {name} full: ok {st}", flush=True)
