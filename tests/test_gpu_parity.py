"""GPU parity: libjdob.so (through its C ABI) against the CPU oracle.

Every case prints its name, shape and entry point before touching the GPU.
Comparison rule: tests/parity.py.
"""

import numpy as np
import pytest

import oracle
from paper_2504_14611_amd import jdob
from paper_2504_14611_amd import workloads as W
from tests.parity import compare

pytestmark = pytest.mark.gpu

THREADS = 16


def _say(label, prob, entry="jdob_solve_batch"):
    print(f"\n[gpu] {label}: {entry} I={W.num_instances(prob)} N={prob['N']} L={prob['L']} "
          f"K={prob['K']} J={prob['J']} {prob['dtype']}", flush=True)


def solve_gpu(prob, label):
    import torch
    _say(label, prob)
    d = jdob.to_device(prob)
    out = jdob.solve_batch(d)
    torch.cuda.synchronize()
    return jdob.to_host(out)


def check(prob, label, tol=1e-5):
    gpu = solve_gpu(prob, label)
    ora = oracle.solve(prob, threads=THREADS)
    st = compare(prob, gpu, ora, tol=tol, label=label)
    print(f"[gpu] {label}: ok {st}", flush=True)
    return gpu, ora


SMALL = [("c0", 256), ("c1", 4096), ("c2", 8192), ("c2b", 4096), ("c3", 4096),
         ("c4", 512), ("c4b", 192)]


@pytest.mark.parametrize("name,n", SMALL)
def test_workload_prefix(name, n):
    check(W.generate(W.WORKLOADS[name], 0, n), f"{name}[:{n}]")


@pytest.mark.parametrize("name", ["c2", "c3", "c4"])
def test_full_size_every_instance(name):
    """The whole batch in the benchmark's launch configuration (no work
    counters), every instance compared with the oracle; a second launch
    with the counters must return the same policy bit for bit, and its
    counters are compared too.  (Every c4 instance is infeasible by the
    workload's definition: about half its users cannot run 50 layers locally
    by a deadline of at most 80 ms, and no batch covering them fits; its
    parity is the status, the counters and the empty policy.)"""
    import torch
    w = W.WORKLOADS[name]
    prob = W.generate(w)
    _say(f"{name} full, every instance", prob)
    d = jdob.to_device(prob)
    gpu = jdob.to_host(jdob.solve_batch(d, counters=False))
    torch.cuda.synchronize()
    cnt = jdob.to_host(jdob.solve_batch(d, counters=True))
    torch.cuda.synchronize()
    del d
    for k, v in gpu.items():
        if v is not None:
            assert np.array_equal(v, cnt[k], equal_nan=True), (name, "counters launch", k)
    gpu["num_feasible"], gpu["num_user_evals"] = cnt["num_feasible"], cnt["num_user_evals"]
    ora = oracle.solve(prob, threads=THREADS)
    st = compare(prob, gpu, ora, label=f"{name} full")
    print(f"[gpu] {name} full: ok {st}", flush=True)


def test_c4b_full_size_sampled():
    """c4b (N = 128, L = 50, every instance feasible with batches of 74 to
    128 users) at full size in the benchmark's launch configuration; the
    oracle, at about 100 instances per second per thread, checks the first
    1024 instances and a seeded sample of 2048 more."""
    w = W.WORKLOADS["c4b"]
    prob = W.generate(w)
    gpu = solve_gpu(prob, "c4b full")
    I = w.num_instances
    rng = np.random.default_rng(23)
    idx = np.unique(np.concatenate([np.arange(1024), rng.choice(np.arange(1024, I), 2048, replace=False)]))
    sub = W.take(prob, idx)
    ora = oracle.solve(sub, threads=THREADS)
    g = {k: (None if v is None else v[idx]) for k, v in gpu.items()}
    st = compare(sub, g, ora, label="c4b full", idx=idx)
    print(f"[gpu] c4b full: ok {st}", flush=True)


def _edge(base, n, stream, **kw):
    return W.generate(W.WORKLOADS[base].replace(name="edge", stream=stream, num_instances=n, **kw))


EDGE_SHAPES = {
    "N1": ("c1", 512, dict(N=1)),
    "N65": ("c4b", 48, dict(N=65, L=12, K=8, J=16)),
    "N127": ("c4b", 32, dict(N=127, L=10, K=8, J=16)),
    "N128": ("c4b", 32, dict(N=128, L=10, K=8, J=16)),
    "N129": ("c4b", 32, dict(N=129, L=10, K=8, J=16)),
    "K1": ("c1", 512, dict(K=1, local_f=(2.0e9, 2.0e9))),
    "J1": ("c1", 512, dict(J=1)),
    "L1": ("c1", 512, dict(L=1)),
    "J100": ("c2b", 256, dict(J=100)),
    "J256": ("c1", 64, dict(J=256, N=8, L=6)),
    "K64": ("c2b", 128, dict(K=64)),
    "N1024": ("c4b", 3, dict(N=1024, L=3, K=4, J=4)),
    "L255": ("c1", 16, dict(L=255, N=4, K=4, J=4, cycles=("lu", 1e5, 2e6))),
    "f64_c1": ("c1", 1024, dict(dtype="f64")),
    "f64_c3": ("c3", 512, dict(dtype="f64")),
    "f64_N70": ("c4b", 16, dict(N=70, L=8, K=8, J=8, dtype="f64")),
    "I1": ("c3", 1, {}),
    "I7": ("c3", 7, {}),
    "I1001": ("c3", 1001, {}),
    # the batch records past N that a pass may read (64 / min(J, 64) of
    # them): GPU level counts that leave idle lanes reading the last one
    "N100_J3": ("c4b", 24, dict(N=100, L=10, K=8, J=3)),
    "N70_J1": ("c4b", 16, dict(N=70, L=8, K=8, J=1)),
    "N33_J63": ("c2b", 64, dict(N=33, L=12, K=8, J=63)),
}


@pytest.mark.parametrize("case", sorted(EDGE_SHAPES))
def test_edge_shapes(case):
    base, n, kw = EDGE_SHAPES[case]
    check(_edge(base, n, 500 + sorted(EDGE_SHAPES).index(case), **kw), case)


def test_empty_batch():
    """A batch of no instances through the binding: every entry point
    returns without launching, and the outputs are empty."""
    import torch
    for name in ("c1", "h1"):
        prob = W.take(W.generate(W.WORKLOADS[name], 0, 4), np.arange(0))
        _say(f"empty batch of {name}", prob, "every entry point")
        d = jdob.to_device(prob)
        outs = [jdob.solve_batch(d), jdob.solve_grouped(d)]
        if name == "c1":
            tab = jdob.eval_user_tables(d)
            outs += [tab, jdob.eval_joint(d, tab)]
        torch.cuda.synchronize()
        for o in outs:
            for k, v in jdob.to_host(o).items():
                assert v is None or v.shape[0] == 0, (name, k)


def test_tied_rates_zero_cycles_zero_bits():
    p = W.generate(W.WORKLOADS["c2b"], 0, 2048)
    p["rate"][:, 1] = p["rate"][:, 0]
    p["rate"][:, 5:9] = p["rate"][:, 4:5]
    p["cycles"][:512, ::3] = 0
    p["bits"][256:1024, 4] = 0
    p["bits"][1024:1536, 0] = 0
    check(p, "ties+zeros")


def test_shared_deadline_ties_everywhere():
    # every user identical: all orders tie, all batches of a size are equal
    p = W.generate(W.WORKLOADS["c1"], 0, 512)
    p["rate"][:] = p["rate"][:, :1]
    p["deadline"][:] = p["deadline"][:, :1]
    check(p, "identical users")


def test_all_infeasible_and_busy_gpu():
    p = W.generate(W.WORKLOADS["c3"], 0, 1024)
    p["deadline"][:512] = np.float32(1e-4)
    rng = np.random.default_rng(5)
    p["t_free"] = rng.uniform(0, 0.1, size=1024).astype(np.float32)
    gpu, ora = check(p, "infeasible+t_free")
    assert (ora["status"][:512] == 1).all()


def _stage_check(prob, name):
    """eval_joint(eval_user_tables(x)) == solve_batch(x) bitwise, and the
    stage-1 tables equal the oracle's bitwise."""
    import torch
    _say(name, prob, "jdob_eval_user_tables + jdob_eval_joint")
    d = jdob.to_device(prob)
    fused = jdob.to_host(jdob.solve_batch(d, freq=True))
    tabs = jdob.eval_user_tables(d)
    joint = jdob.to_host(jdob.eval_joint(d, tabs, freq=True))
    torch.cuda.synchronize()
    tabs = jdob.to_host(tabs)
    for k in fused:
        assert np.array_equal(fused[k], joint[k], equal_nan=True), (name, k)
    ot = oracle.user_tables(prob)
    for k in ot:
        a, b = tabs[k], ot[k]
        if a.dtype.kind == "f":
            it = np.int64 if a.dtype == np.float64 else np.int32
            assert np.array_equal(a.view(it), b.view(it)), (name, k)
        else:
            assert np.array_equal(a, b), (name, k)


def test_stage_parity_and_tables():
    cases = [(W.WORKLOADS[name], n) for name, n in (("c2b", 2048), ("c3", 2048), ("c4b", 64), ("c0", 256))]
    cases.append((W.WORKLOADS["c2b"].replace(name="c2b_J100", stream=590, J=100), 256))
    for w, n in cases:
        _stage_check(W.generate(w, 0, n), w.name)


# Shapes at the edges of the stage-1 walk: a wave covering 64 partition
# points (N = 1), a row longer than the wave (N > 64), runs of only two level
# rows (K = 64), padded level rows (K not a power of two), a single level,
# the longest chain, binary64.
STAGE_SHAPES = {
    "N1_L255_K64": ("c1", 64, dict(N=1, L=255, K=64, J=4, cycles=("lu", 1e5, 2e6))),
    "N3_L40_K17": ("c2b", 128, dict(N=3, L=40, K=17, J=8)),
    "N65_L7_K33_f64": ("c4b", 16, dict(N=65, L=7, K=33, J=8, dtype="f64")),
    "N130_L3_K1": ("c4b", 16, dict(N=130, L=3, K=1, J=8, local_f=(2.0e9, 2.0e9))),
    "N64_L22_K64": ("c3", 64, dict(N=64, K=64)),
    "N33_L9_K5_f64": ("c2b", 128, dict(N=33, L=9, K=5, J=12, dtype="f64")),
    # user counts that are multiples of four (a lane's four entries share a
    # partition point), at every row size 2^0 .. 2^6, with and without pads
    "N4_L8_K1": ("c2b", 128, dict(N=4, L=8, K=1, J=4, local_f=(2.0e9, 2.0e9))),
    "N8_L5_K2_f64": ("c2b", 128, dict(N=8, L=5, K=2, J=4, dtype="f64")),
    "N12_L10_K3": ("c2b", 128, dict(N=12, L=10, K=3, J=8)),
    "N16_L6_K7": ("c2b", 128, dict(N=16, L=6, K=7, J=8)),
    "N20_L13_K64_f64": ("c2b", 64, dict(N=20, L=13, K=64, J=8, dtype="f64")),
    "N128_L50_K33": ("c4b", 16, dict(N=128, L=50, K=33, J=8)),
    # four entries per store, but a lane's entries cross partition points
    "N10_L21_K9": ("c2b", 128, dict(N=10, L=21, K=9, J=8)),
}


@pytest.mark.parametrize("case", sorted(STAGE_SHAPES))
def test_stage_tables_walk_edges(case):
    base, n, kw = STAGE_SHAPES[case]
    _stage_check(_edge(base, n, 640 + sorted(STAGE_SHAPES).index(case), **kw), case)


# Launches long enough for the paired-instance stage-1 kernel (2^18
# instances or more, N a multiple of four, every level row resident, an
# instance's int8 table not whole 128-byte lines); an odd count leaves the
# last workgroup one instance.
PAIRED_SHAPES = {
    "c3_shape": ("c3", dict()),
    "N12_L10_K3": ("c2b", dict(N=12, L=10, K=3, J=8)),
    "N8_L5_K2_f64": ("c2b", dict(N=8, L=5, K=2, J=4, dtype="f64")),
    "N20_L6_K64": ("c2b", dict(N=20, L=6, K=64, J=8)),
}


@pytest.mark.parametrize("case", sorted(PAIRED_SHAPES))
def test_stage_tables_paired_launch(case):
    """Two-stage policy == fused policy bit for bit on every instance, and
    the tables bit for bit equal to the oracle's on the first and last 512
    instances and 1,024 sampled between."""
    import torch
    import bench
    base, kw = PAIRED_SHAPES[case]
    n = (1 << 18) + 1
    w = W.WORKLOADS[base].replace(name="paired", stream=700 + sorted(PAIRED_SHAPES).index(case),
                                  num_instances=n, **kw)
    assert bench.tables_kernel_name(w).startswith("jdob_tables_group_kernel<")
    prob = W.generate(w)
    _say(case, prob, "jdob_eval_user_tables (instances in pairs) + jdob_eval_joint")
    d = jdob.to_device(prob)
    fused = jdob.to_host(jdob.solve_batch(d, freq=True))
    tabs = jdob.eval_user_tables(d)
    joint = jdob.to_host(jdob.eval_joint(d, tabs, freq=True))
    torch.cuda.synchronize()
    tabs = jdob.to_host(tabs)
    for k in fused:
        assert np.array_equal(fused[k], joint[k], equal_nan=True), (case, k)
    rng = np.random.default_rng(11)
    idx = np.unique(np.concatenate([np.arange(512), np.arange(n - 512, n),
                                    rng.integers(512, n - 512, size=1024)]))
    ot = oracle.user_tables(W.take(prob, idx))
    for k in ot:
        a, b = tabs[k][idx], ot[k]
        if a.dtype.kind == "f":
            it = np.int64 if a.dtype == np.float64 else np.int32
            assert np.array_equal(a.view(it), b.view(it)), (case, k)
        else:
            assert np.array_equal(a, b), (case, k)


def test_stage_tables_more_instances_than_one_launch():
    """2^24 + 2^18 + 1 instances with N a multiple of four: both launches of
    the split take instances in pairs (the second from an offset); the
    tables on both sides of the split, at the end and on a seeded sample
    equal the oracle's bit for bit."""
    import torch
    import bench
    n = (1 << 24) + (1 << 18) + 1
    w = W.WORKLOADS["c1"].replace(name="split", stream=779, num_instances=n, N=4, L=2, K=2, J=2)
    assert bench.tables_kernel_name(w) == "jdob_tables_group_kernel<float, 1, 2>"
    prob = W.generate(w)
    _say("2^24 + 2^18 + 1 instances", prob, "jdob_eval_user_tables")
    tabs = jdob.eval_user_tables(jdob.to_device(prob))
    torch.cuda.synchronize()
    rng = np.random.default_rng(23)
    idx = np.unique(np.concatenate([np.arange(0, 64), np.arange((1 << 24) - 64, (1 << 24) + 64),
                                    np.arange(n - 64, n), rng.choice(n, 4000, replace=False)]))
    ti = torch.as_tensor(idx, device="cuda")
    got = {k: v[ti].cpu().numpy() for k, v in tabs.items()}
    ot = oracle.user_tables(W.take(prob, idx))
    for k in ot:
        a, b = got[k], ot[k]
        if a.dtype.kind == "f":
            assert np.array_equal(a.view(np.int32), b.view(np.int32)), k
        else:
            assert np.array_equal(a, b), k
    print(f"[gpu] 2^24 + 2^18 + 1 instances: tables ok on {idx.size} instances", flush=True)


def test_stage_tables_unaligned_destination():
    """Tables written through pointers one element past a 16-byte boundary
    (element stores instead of the four-entry stores) equal the aligned
    ones bit for bit."""
    import torch
    prob = W.generate(W.WORKLOADS["c3"], 0, 257)
    _say("c3[:257] tables at unaligned pointers", prob, "jdob_eval_user_tables")
    d = jdob.to_device(prob)
    a = jdob.eval_user_tables(d)
    big = {k: torch.empty((v.numel() + 16,), dtype=v.dtype, device=v.device) for k, v in a.items()}
    b = {k: big[k][1:1 + v.numel()].view(v.shape) for k, v in a.items()}
    jdob.eval_user_tables(d, out=b)
    torch.cuda.synchronize()
    for k in a:
        x, y = a[k].cpu().numpy(), b[k].cpu().numpy()
        if x.dtype.kind == "f":
            x, y = x.view(np.int32), y.view(np.int32)
        assert np.array_equal(x, y), k


def test_deterministic_and_chunkable():
    import torch
    prob = W.generate(W.WORKLOADS["c3"], 0, 5000)
    _say("c3 determinism/chunks", prob)
    d = jdob.to_device(prob)
    a = jdob.to_host(jdob.solve_batch(d, freq=True))
    b = jdob.to_host(jdob.solve_batch(d, freq=True))
    torch.cuda.synchronize()
    for k in a:
        assert np.array_equal(a[k], b[k], equal_nan=True), k
    # the launch without the optional work counters returns the same policy
    c = jdob.to_host(jdob.solve_batch(d, counters=False))
    torch.cuda.synchronize()
    for k in a:
        if c[k] is not None:
            assert np.array_equal(a[k], c[k], equal_nan=True), ("no counters", k)
    # solving sub-ranges through offset pointers gives the same rows
    for lo, hi in ((0, 1), (1, 4000), (4000, 5000), (777, 2777)):
        sub = {k: (v[lo:hi] if k in ("cycles", "bits", "alpha", "beta", "rate", "deadline", "t_free")
                   else v) for k, v in d.items()}
        c = jdob.to_host(jdob.solve_batch(sub, freq=True))
        torch.cuda.synchronize()
        for k in a:
            assert np.array_equal(a[k][lo:hi], c[k], equal_nan=True), (lo, hi, k)


def test_more_instances_than_one_launch():
    """2^24 + 5 instances: the library splits the batch into launches of at
    most 2^24 workgroups; the instances on both sides of the split and a
    seeded sample are checked against the oracle."""
    import torch
    n = (1 << 24) + 5
    prob = _edge("c1", n, 777, N=2, L=2, K=2, J=2)
    _say("2^24 + 5 instances", prob)
    gpu = jdob.to_host(jdob.solve_batch(jdob.to_device(prob), counters=True))
    torch.cuda.synchronize()
    rng = np.random.default_rng(19)
    idx = np.unique(np.concatenate([np.arange(0, 64), np.arange((1 << 24) - 64, n),
                                    rng.choice(n, 4000, replace=False)]))
    sub = W.take(prob, idx)
    ora = oracle.solve(sub, threads=THREADS)
    g = {k: (None if v is None else v[idx]) for k, v in gpu.items()}
    st = compare(sub, g, ora, label="2^24 + 5", idx=idx)
    print(f"[gpu] 2^24 + 5 instances: ok {st}", flush=True)
