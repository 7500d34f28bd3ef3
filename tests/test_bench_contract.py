"""The benchmark's command line and JSON line (bench.py).

CPU: the host-side pieces of bench.py (search-mode names, family sizes,
algorithmic bytes) against their definitions, and the refusal of more than
one GPU.  GPU: one short run of bench.py whose JSON line must carry every
field of the contract with consistent values.
"""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2504_14611_amd import workloads as W  # noqa: E402


def test_mode_names_round_trip():
    for bits in range(16):
        assert bench.parse_mode(bench.mode_text(bits)) == bits
    assert bench.parse_mode("grid") == 0
    assert bench.parse_mode("greedy+continuous") == 9
    with pytest.raises(SystemExit):
        bench.parse_mode("fastest")


def test_family_sizes():
    w = W.WORKLOADS["c3"]
    assert bench.family_size(w, 0) == 22 * 32 * 32 + 1       # every (s, j, b) and LC
    assert bench.family_size(w, 1) == 22 * 32 + 1            # one batch per (s, j)
    assert bench.family_size(w, 2) == 22 * 32 + 1            # top GPU level only
    assert bench.family_size(w, 4) == 32 * 32 + 1            # s = 0 only
    assert bench.family_size(w, 7) == 1 + 1
    g = W.WORKLOADS["g10"]
    # every group of consecutive users in deadline order is solved once
    assert bench.grouped_family_size(g, 0) == sum(
        (22 * 32 * n + 1) * (10 - n + 1) for n in range(1, 11))


def test_algorithmic_bytes():
    w = W.WORKLOADS["c3"]
    ins, outs = bench.algorithmic_bytes(w)
    assert ins == w.num_instances * (4 * 22 + 2 + 2 * 32) * 4   # 616 B per instance
    assert outs == w.num_instances * (16 + 2 * 4 + 2 * 32)      # 88 B per instance


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


KEYS = {"metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
        "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"}


@pytest.mark.gpu
def test_bench_json_line():
    print("\n[gpu] bench.py --workload c1 --steps 3 --warmup 1 --cpu-sample 256", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "c1",
                        "--steps", "3", "--warmup", "1", "--cpu-sample", "256"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    d = json.loads(lines[0])
    assert KEYS <= set(d)
    w = W.WORKLOADS["c1"]
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["unit"] == "candidates/s" and d["higher_is_better"] is True
    assert d["config"]["workload"].startswith("c1:") and d["config"]["instances"] == w.num_instances
    # value is the whole batch's candidates over the wall time per step
    cands = w.num_instances * bench.family_size(w, 0)
    assert abs(d["value"] - cands / (d["ms_per_step"] * 1e-3)) <= 1e-6 * d["value"]
    rf = d["roofline"]
    assert rf["bound"] == "alu" and rf["unit"] == "TOP/s"
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-9
    assert 0 <= rf["frac"] <= 1
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] == 1 and cb["value"] > 0
    assert "256" in cb["sample"]
    ps = d["parity_sample"]
    assert ps["status_mismatch"] == 0 and ps["counter_mismatch"] == 0
    t1 = d["stages"]["jdob_eval_user_tables"]
    assert t1["kernel"] == bench.tables_kernel_name(w) and t1["ms"] > 0
    assert (t1["read_bytes"], t1["write_bytes"]) == bench.stage_bytes(w)
    assert 0 < t1["hbm_frac"] <= 1 and d["stages"]["jdob_eval_joint"]["ms"] > 0
    e2e = d["end_to_end"]
    assert e2e["serial"]["ms"] > 0 and e2e["pipelined"]["chunks"] in bench.E2E_PIECES


def test_stage1_kernel_choice():
    """The stage-1 kernel bench.py names for each workload: pairs of
    instances per workgroup only on long launches whose instance rows are all
    resident and whose int8 tables are not whole 128-byte lines."""
    from paper_2504_14611_amd import workloads as W
    want = {"c0": "jdob_tables_kernel<double, true, 2>", "c1": "jdob_tables_kernel<float, true, 3>",
            "c2": "jdob_tables_kernel<float, true, 4>", "c3": "jdob_tables_group_kernel<float, 4, 2>",
            "c4": "jdob_tables_kernel<float, true, 5>", "c4b": "jdob_tables_kernel<float, true, 5>"}
    for k, v in want.items():
        assert bench.tables_kernel_name(W.WORKLOADS[k]) == v, k
    w = W.WORKLOADS["c3"].replace(num_instances=(1 << 18) - 1)
    assert bench.tables_kernel_name(w) == "jdob_tables_kernel<float, true, 4>"
    w = W.WORKLOADS["c3"].replace(N=10)  # (L+1)*N = 230: not four-entry rows of one point
    assert bench.tables_kernel_name(w) == "jdob_tables_kernel<float, false, -1>"
