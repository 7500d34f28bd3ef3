"""GPU parity over seeded random shapes and search modes, against the oracle.

The other GPU tests pin chosen shapes: the workloads, their edges, the
limits.  Here each case draws (N, L, K, J, mode, precision) from a seeded
generator, so the kernels' shape-dependent paths (user counts that are not
a multiple of the four- and eight-user steps of the user loop, level rows
with and without padding, GPU levels beyond one wave, partial passes) are
met in combinations nobody chose.  The inputs keep the distributions of a
base workload, alternating between bases where offloading wins for some
users (c2b, h2 with Table I's parameters), for all of them or none (p4a,
Table I) or rarely (h1), so that the argmin is decided among offloading
candidates as well as against local computing; the groupings use p5 and
h5 (Table I, most instances offload in some group).
A further category draws more than 64 users, and another runs the
two-stage calls (the stage-1 tables bit for bit against the oracle's, the
two-stage policy against the fused one).  Comparison rules:
tests/parity.py, compare_grouped in
tests/test_gpu_grouped.py.  Every case prints its draw before touching the
GPU.
"""

import numpy as np
import pytest

from tests.test_gpu_hetero import check as hetero_check
from tests.test_gpu_parity import _edge, check

pytestmark = pytest.mark.gpu

MODES = (0, 1, 2, 3, 4, 8, 9, 10, 12)


def draw(seed, n_max, l_max, k_max, j_max):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(1, n_max + 1))
    L = int(rng.integers(1, l_max + 1))
    K = int(rng.integers(2, k_max + 1))
    J = int(rng.integers(1, j_max + 1))
    mode = int(rng.choice(MODES))
    dtype = "f64" if rng.random() < 0.2 else "f32"
    return N, L, K, J, mode, dtype


def problem(base, seed, n_inst, N, L, K, J, mode, dtype):
    p = _edge(base, n_inst, seed, N=N, L=L, K=K, J=J, dtype=dtype)
    p["mode"] = mode
    return p


@pytest.mark.parametrize("k", range(24))
def test_random_shapes_shared_parameters(k):
    N, L, K, J, mode, dtype = draw(7000 + k, 64, 30, 64, 160)
    label = f"random {k}: N={N} L={L} K={K} J={J} mode={mode} {dtype}"
    check(problem("c2b" if k % 2 == 0 else "p4a", 7000 + k, 96, N, L, K, J, mode, dtype), label)


# More users than one wave (user rows in several chunks) with GPU level
# counts that do not divide 64, so that some lanes of every pass hold no
# (j, b) pair and must read an infeasible record: with N > 64 the index
# b0 + 64 is a real batch record.  Seeds 30, 73, 100 and 108 draw such
# shapes (J = 51, 37, 56, 36).
@pytest.mark.parametrize("k", [30, 73, 100, 108] + list(range(16)))
def test_random_shapes_many_users(k):
    N, L, K, J, mode, dtype = draw(30000 + k, 300, 16, 64, 256)
    N = max(N, 65)
    label = f"random many users {k}: N={N} L={L} K={K} J={J} mode={mode} {dtype}"
    check(problem("c2b" if k % 2 == 0 else "p4a", 30000 + k, 48, N, L, K, J, mode, dtype), label)


@pytest.mark.parametrize("k", range(12))
def test_random_shapes_heterogeneous(k):
    N, L, K, J, mode, dtype = draw(7100 + k, 64, 24, 24, 96)
    label = f"random hetero {k}: N={N} L={L} K={K} J={J} mode={mode} {dtype}"
    hetero_check(problem("h2" if k % 2 == 0 else "h1", 7100 + k, 64, N, L, K, J, mode, dtype), label)


@pytest.mark.parametrize("k", range(8))
def test_random_shapes_grouped(k):
    from tests.test_gpu_grouped import check as grouped_check
    N, L, K, J, mode, dtype = draw(7200 + k, 14, 14, 16, 40)
    label = f"random grouped {k}: N={N} L={L} K={K} J={J} mode={mode} {dtype}"
    p = problem("p5", 7200 + k, 32, N, L, K, J, mode, dtype)
    grouped_check(p, label, freq=True)


@pytest.mark.parametrize("k", range(6))
def test_random_shapes_heterogeneous_grouped(k):
    from tests.test_gpu_grouped import check as grouped_check
    N, L, K, J, mode, dtype = draw(7300 + k, 12, 12, 12, 32)
    label = f"random hetero grouped {k}: N={N} L={L} K={K} J={J} mode={mode} {dtype}"
    p = problem("h5", 7300 + k, 24, N, L, K, J, mode, dtype)
    grouped_check(p, label, freq=True)


@pytest.mark.parametrize("k", range(12))
def test_random_shapes_two_stage(k):
    from tests.test_gpu_parity import _stage_check
    N, L, K, J, mode, dtype = draw(7400 + k, 160, 64, 64, 96)
    label = f"random two-stage {k}: N={N} L={L} K={K} J={J} mode={mode} {dtype}"
    _stage_check(problem("c2b" if k % 2 == 0 else "p4a", 7400 + k, 32, N, L, K, J, mode, dtype), label)
