"""GPU-vs-oracle comparison rule (test helper).

Per instance:
* status, and the integer work counters (feasible candidates, sum of b over
  them) are equal;
* the chosen candidate (cut, GPU level, batch) is equal, unless the oracle's
  two best energies are within `tol` of each other; then the GPU's choice
  must be a feasible candidate whose oracle energy is within `tol` of the
  oracle's minimum;
* with the same candidate, every per-user level, frequency (when the GPU
  returned them) and offload flag, the release time and the energy
  (re-summed in the fixed order of the ABI) are bitwise equal: every
  operation on the path is pinned;
* the energy is within `tol` (relative) of the oracle's in every case.
"""

import numpy as np

import oracle

TOL = 1e-5


def _in_family(prob, r, gpu, label):
    """A near-tie swap must still be a candidate of the problem's search
    mode: s = 0 or local computing with binary offloading, the top GPU level
    without edge DVFS, and with greedy batching a batch that cannot grow."""
    mode = int(prob.get("mode", 0))
    s, j, b = int(gpu["cut"][r]), int(gpu["gpu_level"][r]), int(gpu["batch"][r])
    if s == prob["L"]:
        return
    if mode & oracle.MODE_BINARY:
        assert s == 0, f"{label}: binary offloading picked s = {s}"
    if mode & oracle.MODE_FIXED_EDGE:
        assert j == prob["J"] - 1, f"{label}: fixed edge frequency picked j = {j}"
    if mode & oracle.MODE_GREEDY and b < prob["N"]:
        assert not oracle.eval_candidate(prob, int(r), s, j, b + 1)["feasible"], \
            f"{label}: greedy batch {b} at ({s}, {j}) could grow"


def compare(prob, gpu, ora, tol=TOL, idx=None, label=""):
    """gpu/ora: dicts of host arrays; idx: instance numbers of `prob` rows
    (defaults to 0..I-1) used for near-tie candidate re-evaluation."""
    I = len(ora["status"])
    if idx is None:
        idx = np.arange(I)
    st = {"instances": I, "feasible": int((ora["status"] == 0).sum()), "near_ties": 0,
          "tie_swaps": 0}
    assert np.array_equal(gpu["status"], ora["status"]), label + " status"
    if gpu.get("num_feasible") is not None:
        bad = np.nonzero(gpu["num_feasible"] != ora["num_feasible"])[0]
        assert bad.size == 0, f"{label} num_feasible differs at {bad[:5]}"
        bad = np.nonzero(gpu["num_user_evals"] != ora["num_user_evals"])[0]
        assert bad.size == 0, f"{label} num_user_evals differs at {bad[:5]}"
    feas = ora["status"] == 0
    inf = ~feas
    assert np.isinf(gpu["energy"][inf]).all() and np.isinf(gpu["t_free_out"][inf]).all()
    assert (gpu["cut"][inf] == -1).all() and (gpu["user_level"][inf] == -1).all()
    freq = gpu.get("user_freq") is not None
    if freq:
        assert (gpu["user_freq"][inf] == 0).all(), label + " user_freq of infeasible instances"
    e_or = ora["energy"].astype(np.float64)
    e_gp = gpu["energy"].astype(np.float64)
    rel = np.abs(e_gp[feas] - e_or[feas]) / np.maximum(np.abs(e_or[feas]), 1e-300)
    assert (rel <= tol).all(), f"{label} energy rel err {rel.max()}"
    same = feas & (gpu["cut"] == ora["cut"]) & (gpu["gpu_level"] == ora["gpu_level"]) & \
        (gpu["batch"] == ora["batch"])
    with np.errstate(invalid="ignore"):
        near = (ora["energy_second"].astype(np.float64) - e_or) <= tol * np.abs(e_or)
    st["near_ties"] = int((feas & near).sum())
    diff = np.nonzero(feas & ~same)[0]
    for r in diff:
        assert near[r], (f"{label} instance {idx[r]}: gpu {(gpu['cut'][r], gpu['gpu_level'][r], gpu['batch'][r])}"
                         f" oracle {(ora['cut'][r], ora['gpu_level'][r], ora['batch'][r])}"
                         f" E {e_gp[r]} vs {e_or[r]} second {ora['energy_second'][r]}")
        c = oracle.eval_candidate(prob, int(r), int(gpu["cut"][r]), int(gpu["gpu_level"][r]),
                                  int(gpu["batch"][r]))
        assert c["feasible"], f"{label} instance {idx[r]}: GPU picked an infeasible candidate"
        _in_family(prob, r, gpu, label)
        assert abs(c["energy"] - e_or[r]) <= tol * abs(e_or[r])
        assert np.array_equal(gpu["user_level"][r], c["user_level"])
        assert np.array_equal(gpu["user_offload"][r], c["user_offload"])
        if freq:
            assert np.array_equal(_bits(gpu["user_freq"][r]), _bits(c["user_freq"]))
        st["tie_swaps"] += 1
    for k in ("user_level", "user_offload"):
        bad = np.nonzero((gpu[k][same] != ora[k][same]).any(axis=1))[0]
        assert bad.size == 0, f"{label} {k} differs at {idx[np.nonzero(same)[0][bad[:5]]]}"
    for k in ("t_free_out", "energy"):
        a, b = gpu[k][same], ora[k][same]
        bad = np.nonzero(_bits(a) != _bits(b))[0]
        assert bad.size == 0, f"{label} {k} not bitwise equal at {idx[np.nonzero(same)[0][bad[:5]]]}"
    if freq:
        bad = np.nonzero((_bits(gpu["user_freq"][same]) != _bits(ora["user_freq"][same])).any(axis=1))[0]
        assert bad.size == 0, f"{label} user_freq differs at {idx[np.nonzero(same)[0][bad[:5]]]}"
    return st


def _bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.int64 if a.dtype == np.float64 else np.int32)
