#!/usr/bin/env python3
"""Benchmark of batched J-DOB policy evaluation on one MI355X.

One step = one jdob_solve_batch over the whole batch of the workload (all
stages: instance sums, rate order, batch deadlines, per-partition-point
rows, the candidate grid with deadline masking, per-user levels and energy,
the argmin and the winner's policy), with the inputs resident in HBM.

Prints ONE JSON line:
  value   = candidate policies evaluated per second (every (s, j, b) of
            L*J*N plus local computing counts once its feasibility is decided)
  roofline: the solve kernel against the FP32 VALU issue rate (it is a loop
            of compares, selects and adds: no dense contraction, and HBM
            traffic is ~1 KB per instance); "achieved" counts the method's
            algorithmic operations (14 per feasible candidate, 2 +
            ceil(log2(K+1)) per offloader evaluation), "useful_work" the
            stricter count of what this kernel cannot avoid, and
            valu_busy_counter the measured fraction of VALU issue slots
            used (SQ_ACTIVE_INST_VALU less the dual-issue slots), with the
            counter-classified FP32/INT32 lane-op rates in valu_counters
  cpu_baseline: the CPU oracle, single thread pinned to one core, on a
            bounded sample (and, secondary, the same sample on up to 16
            threads).
  end_to_end: the same batch held in pinned host memory, copied in and the
            policy copied out around the solve (PCIe-inclusive; not "value"),
            in sequence and pipelined over three streams (2, 4 or 8 pieces,
            the fastest reported).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X: 256 CUs x 4 SIMD x 16 lanes x 2.4 GHz = 39.32e12 non-packed 32-bit
# VALU lane-operations per second.
VALU_PEAK_OPS = 256 * 4 * 16 * 2.4e9
HBM_PEAK = 8.0e12
# Algorithmic lane-operations of the method (the roofline's "achieved"),
# for the work the kernel evaluates candidate by candidate:
#   per feasible candidate: batch latency 3, slack 1, the three tests 4, GPU
#   energy 1, total 2-3, argmin 2 = 14;
#   per offloader evaluation of a feasible candidate: the budget subtract, a
#   search of its lowest fitting level among K (ceil(log2(K+1)) compares)
#   and the energy add; with a continuous CPU frequency: subtract,
#   reciprocal, multiply, clamp below, clamp above, square-and-add = 6.
# Infeasible candidates are decided in bulk (a partition point that fails at
# its most favourable candidate, a pass with no feasible lane); charging 14
# to each of them would put "achieved" above the peak (c4: 25x).
OPS_PER_CANDIDATE = 14
OPS_PER_USER_EVAL_CONT = 6
# The stricter count of the work this kernel cannot avoid ("useful work"):
# 16 per feasible candidate (infeasible ones are mostly decided in bulk) and
# 3 per offloader evaluation (subtract, one compare against the lane's
# current level, add: the levels only move up along the users); with
# heterogeneous users the level is searched in each user's own table.
USEFUL_PER_FEASIBLE_CAND = 16
USEFUL_PER_USER_EVAL = 3


def model_ops_per_user_eval(w, mode) -> int:
    if mode & MODE_BITS["continuous"]:
        return OPS_PER_USER_EVAL_CONT
    return 2 + int(np.ceil(np.log2(w.K + 1)))


def useful_ops_per_user_eval(w, mode) -> int:
    if mode & MODE_BITS["continuous"]:
        return OPS_PER_USER_EVAL_CONT
    if w.users is not None:
        return 2 + int(np.ceil(np.log2(w.K + 1)))
    return USEFUL_PER_USER_EVAL


def log(*a):
    print(*a, file=sys.stderr, flush=True)


KERNEL_SRC = tuple(os.path.join(ROOT, "paper_2504_14611_amd", "csrc", f)
                   for f in ("jdob.hip", "jdob_hetero.hip", "jdob_common.h")) + (
    os.path.join(ROOT, "include", "jdob.h"),)


def source_hash() -> str:
    """First 16 hex digits of sha256 over the kernel sources and the header
    with comments and white space removed: an edit of the code changes it,
    an edit of a comment does not."""
    h = hashlib.sha256()
    for path in KERNEL_SRC:
        src = open(path).read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update("".join(src.split()).encode())
    return h.hexdigest()[:16]


def measured_counters(kernel: str, tag: str) -> dict:
    """Figures from the committed rocprofv3 counter summary of this kernel,
    workload and mode (HBM bytes per launch; VALU busy fraction, dual-issue
    fraction, VALU instructions per issue slot, FP32 and INT32 lane-op
    rates), or {} if it is missing or was taken on other kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{tag}_traffic.txt")
    if not os.path.exists(path):
        return {}
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256_16") != source_hash():
        return {}
    def num(k):
        return float(kv[k]) if k in kv else None
    return {"traffic": num("hbm_bytes_per_launch"),
            "valu": {"busy": num("valu_busy_fraction"),
                     "dual_issue": num("valu_dual_issue_fraction"),
                     "instructions_per_slot": num("valu_instructions_per_slot"),
                     "fp32_lane_ops_per_s": num("fp32_lane_ops_per_s"),
                     "int32_lane_ops_per_s": num("int32_lane_ops_per_s")}}


MODE_BITS = {"grid": 0, "greedy": 1, "fixed-edge": 2, "binary": 4, "continuous": 8}


def mode_text(bits: int) -> str:
    names = [k for k, v in MODE_BITS.items() if v and bits & v]
    return "+".join(names) if names else "grid"


def parse_mode(text: str) -> int:
    """'grid', or '+'-joined names among greedy, fixed-edge, binary,
    continuous."""
    bits = 0
    for part in text.split("+"):
        if part not in MODE_BITS:
            raise SystemExit(f"bench.py: unknown mode {part!r} (choose from {sorted(MODE_BITS)})")
        bits |= MODE_BITS[part]
    return bits


def family_size(w, mode: int) -> int:
    """Candidates per instance in the searched family: every (s, j, b) or
    one greedy b per (s, j), over the searched s and j, plus local computing."""
    Ls = 1 if mode & MODE_BITS["binary"] else w.L
    Js = 1 if mode & MODE_BITS["fixed-edge"] else w.J
    return Ls * Js * (1 if mode & MODE_BITS["greedy"] else w.N) + 1


def algorithmic_bytes(w, grouped=False, freq=False):
    """HBM bytes one timed launch must move: per instance the inputs
    cycles[L], bits[L+1], alpha[L], beta[L], rate[N], deadline[N], t_free and
    the outputs -- status, cut, gpu_level, batch (int32), energy, t_free_out
    and user_level[N], user_offload[N] (int8) for one solve; status,
    num_groups, energy, t_free_out, and per user order, group_end (int16),
    group_cut, group_gpu_level, group_batch (int32), group_energy,
    group_t_free, user_level, user_offload, user_group (int8) for the
    grouping; with a continuous CPU frequency also user_freq[N]; with
    heterogeneous users also zeta, kappa, p_tx [N] and the levels [N][K].
    The timed launches fill no work counters."""
    sz = 8 if w.dtype == "f64" else 4
    I, N, L = w.num_instances, w.N, w.L
    uf = N * sz if freq else 0
    users = N * (3 + w.K) * sz if w.users is not None else 0
    inputs = I * ((4 * L + 2 + 2 * N) * sz + users)
    if grouped:
        return inputs, I * (8 + 2 * sz + N * (2 + 2 + 12 + 2 * sz + 3) + uf)
    return inputs, I * (16 + 2 * sz + 2 * N + uf)


def stage_bytes(w):
    """HBM bytes of one stage-1 launch (jdob_eval_user_tables): per instance
    it reads cycles [L], bits [L+1], rate and deadline [N] (the GPU
    coefficients alpha and beta do not enter the tables), and writes the rate
    order [N] (int16), the batch deadlines [N], the minimum batch (int32)
    and, per (partition point, user), the upload time, gamma, the user's own
    energy and slack and its level (int8)."""
    sz = 8 if w.dtype == "f64" else 4
    I, N, L = w.num_instances, w.N, w.L
    return I * (2 * L + 1 + 2 * N) * sz, I * (2 * N + N * sz + 4 + (L + 1) * N * (4 * sz + 1))


def time_stages(w, d, host, steps, warmup, stream):
    """The two-stage entry points on the same batch, after the timed region:
    event times of jdob_eval_user_tables (HBM-bound: its tables are the
    largest arrays of the path) and of jdob_eval_joint, both launched on the
    current stream, whose events are recorded on `stream`; the two-stage
    policy must equal the fused call's bit for bit."""
    import torch
    from paper_2504_14611_amd import jdob
    tab = jdob.eval_user_tables(d)
    out = jdob.alloc_policy(d, counters=False)
    for _ in range(warmup):
        jdob.eval_user_tables(d, tab)
        jdob.eval_joint(d, tab, out)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    for e in ev:
        e[0].record(stream)
        jdob.eval_user_tables(d, tab)
        e[1].record(stream)
        jdob.eval_joint(d, tab, out)
        e[2].record(stream)
    torch.cuda.synchronize()
    joint = jdob.to_host(out)
    for k, v in joint.items():
        if v is not None:
            assert np.array_equal(v, host[k], equal_nan=True), f"two-stage call differs in {k}"
    t1 = float(np.mean([a.elapsed_time(b) for a, b, _ in ev]))
    t2 = float(np.mean([b.elapsed_time(c) for _, b, c in ev]))
    rd, wr = stage_bytes(w)
    assert wr == sum(v.numel() * v.element_size() for v in tab.values()), "stage-1 byte model"
    T = "double" if w.dtype == "f64" else "float"
    del tab
    return {"jdob_eval_user_tables": {
                "kernel": tables_kernel_name(w), "ms": t1, "read_bytes": rd, "write_bytes": wr,
                "hbm_achieved_GBps": (rd + wr) / (t1 * 1e-3) / 1e9,
                "hbm_frac": (rd + wr) / (t1 * 1e-3) / HBM_PEAK},
            "jdob_eval_joint": {"ms": t2},
            "steps": steps}


# Workloads solved with the outer grouping (jdob_solve_grouped); the others
# with jdob_solve_batch.
GROUPED = {"g10", "g20", "p5", "h5"}
# CPU-baseline sample per workload: about 15 s of single-threaded oracle time
CPU_SAMPLE = {"c0": 256, "c1": 4096, "c2": 65536, "c2b": 65536, "c3": 65536, "c4": 32768,
              "c4b": 1536, "g10": 8192, "g20": 1024, "p4a": 65536, "p4b": 65536, "p5": 16384,
              "h1": 65536, "h2": 65536, "h5": 32768}
CPU_SAMPLE_DEFAULT = 4096
# Threads of the secondary (multi-threaded) oracle timing: at most the
# cores one GPU's share of a multi-GPU host offers
MAX_ORACLE_THREADS = 16
# Host-resident batches: timed batches per piece count, and the piece counts
# of the pipelined version (the fastest is reported, with all of them)
E2E_STEPS = 5
E2E_PIECES = (2, 4, 8)


def grouped_family_size(w, mode: int) -> int:
    """Candidates the grouping program evaluates per instance: the family of
    every group ord[j..i-1] it solves, j < i <= N."""
    return sum(family_size(w.replace(N=g), mode) * (w.N - g + 1) for g in range(1, w.N + 1))


def host_cpu():
    """Model name of the host CPU and the cores this process may run on."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, sorted(os.sched_getaffinity(0))


def _tables_layout(N, L, K, szT):
    """(row-size exponent lg, partition points per resident run, LDS bytes of
    one instance): the stage-1 LDS layout of the library (make_tlayout)."""
    a8 = lambda x: (x + 7) & ~7
    o = 0
    for b in (L * szT, (L + 1) * szT, (L + 1) * szT, K * szT, K * szT):
        o = a8(o + b)
    for b in (N * szT, N * szT):  # rates, deadlines: 4-entry aligned
        o = (o + 4 * szT - 1) & ~(4 * szT - 1)
        o = a8(o + b)
    o = a8(o + (N + 1) * 8)
    o = a8(o + N * 4)
    lg = 0
    while (1 << lg) < K:
        lg += 1
    rowb = (1 << lg) * 2 * szT
    run = 4096 // rowb
    run = L + 1 if run >= L + 1 else run & ~3
    o = (o + 15) & ~15
    return lg, run, o + run * rowb


def tables_kernel_name(w) -> str:
    """The stage-1 kernel the library launches for workload w (the rule of
    its launch code): four-entry stores when every instance's rows start on
    a 16-byte boundary; with N a multiple of four the variant for level rows
    of 2^lg entries, and pairs of instances per workgroup when the launch is
    long (2^18 instances or more), an instance's rows are all resident, two
    instances' LDS fit a workgroup and the int8 table of an instance is not
    whole 128-byte lines."""
    T = "double" if w.dtype == "f64" else "float"
    szT = 8 if w.dtype == "f64" else 4
    E = (w.L + 1) * w.N
    vec = E % 4 == 0
    lg, run, total = _tables_layout(w.N, w.L, w.K, szT)
    if vec and w.N % 4 == 0:
        n = min(w.num_instances, 1 << 24)
        if (n >= 1 << 18 and run >= w.L + 1 and E % 128 != 0
                and 2 * ((total + 15) & ~15) <= 64 * 1024):
            return f"jdob_tables_group_kernel<{T}, {lg}, 2>"
        return f"jdob_tables_kernel<{T}, true, {lg}>"
    return f"jdob_tables_kernel<{T}, {'true' if vec else 'false'}, -1>"


def cpu_baseline(prob, w, sample, cand_per_inst, grouped):
    """The oracle on the first `sample` instances: single-threaded and pinned
    to one core (the baseline), then on up to MAX_ORACLE_THREADS threads
    (secondary; the same results)."""
    import oracle
    from paper_2504_14611_amd import workloads as W
    sub = W.take(prob, np.arange(sample))
    run = oracle.solve_grouped if grouped else oracle.solve
    model, cores = host_cpu()
    os.sched_setaffinity(0, {cores[0]})
    try:
        # in eight pieces, a progress line after each (a long quiet run
        # would look hung to a watcher)
        parts, dt = [], 0.0
        bounds = np.linspace(0, sample, 9).astype(int)
        for a, b in zip(bounds[:-1], bounds[1:]):
            if b <= a:
                continue
            piece = W.take(sub, np.arange(a, b))
            t0 = time.perf_counter()
            parts.append(run(piece, threads=1))
            dt += time.perf_counter() - t0
            log(f"[bench] CPU oracle: {b}/{sample} instances, {dt:.1f} s")
        o = {k: (None if parts[0][k] is None else np.concatenate([q[k] for q in parts]))
             for k in parts[0]}
    finally:
        os.sched_setaffinity(0, set(cores))
    nth = min(len(cores), MAX_ORACLE_THREADS)
    t0 = time.perf_counter()
    om = run(sub, threads=nth)
    dtm = time.perf_counter() - t0
    for k in ("status", "energy"):
        assert np.array_equal(o[k], om[k], equal_nan=True), f"threaded oracle differs in {k}"
    cand = sample * cand_per_inst
    what = "jo_solve_grouped" if grouped else "jo_solve"
    return o, {"value": cand / dt, "unit": "candidates/s", "cores": 1, "kind": "oracle",
               "seconds": dt, "instances_per_s": sample / dt,
               "sample": f"first {sample} instances of workload {w.name} "
                         f"({cand} candidates), single-threaded C oracle ({what}) pinned to one core",
               "host": {"cpu": model, "cores_available": len(cores)},
               "threads": {"threads": nth, "seconds": dtm, "value": cand / dtm,
                           "instances_per_s": sample / dtm}}


def end_to_end(prob, d, alloc, solve, steps, chunk_counts):
    """Host-resident batch: pinned host inputs copied to the device, solved,
    and the policy copied back into pinned host arrays.  Returns the wall ms
    per batch for each piece count, the bytes each way, and each run's host
    outputs.

    1 piece runs copy-in, solve, copy-out in sequence on one stream.  More
    pieces split the instance range (offset pointers: instances are
    independent) and pipeline them over three streams, one for host-to-device
    copies, one for the solves and one for device-to-host copies, chained by
    events: piece c+1 is copied in and piece c-1 copied out while piece c is
    solved.  Pipelining pays where the copies are comparable to the kernel;
    where a piece holds too few instances to keep the GPU busy between its
    first and last wave, the pieces' ragged ends cost more than it saves."""
    import torch
    shared = ("local_freq", "gpu_freq")
    per_inst = [k for k, v in d.items() if torch.is_tensor(v) and k not in shared]
    hin = {}
    for k in per_inst:
        hin[k] = torch.empty(d[k].shape, dtype=d[k].dtype, pin_memory=True)
        hin[k].copy_(torch.from_numpy(np.ascontiguousarray(prob[k])))
    dd = dict(d)
    for k in per_inst:
        dd[k] = torch.empty_like(d[k])
    out = alloc(dd, counters=False)
    outs = [k for k, v in out.items() if v is not None]
    hout = {k: torch.empty(out[k].shape, dtype=out[k].dtype, pin_memory=True) for k in outs}
    s_one = torch.cuda.current_stream()
    s_in, s_run, s_out = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    I = int(d["rate"].shape[0])
    torch.cuda.synchronize()

    def one(chunks):
        cuts = np.linspace(0, I, chunks + 1).astype(np.int64)
        ci, cr, co = (s_one, s_one, s_one) if chunks == 1 else (s_in, s_run, s_out)
        for c in range(chunks):
            a, b = int(cuts[c]), int(cuts[c + 1])
            with torch.cuda.stream(ci):
                for k in per_inst:
                    dd[k][a:b].copy_(hin[k][a:b], non_blocking=True)
            cr.wait_stream(ci)
            sub = dict(dd)
            for k in per_inst:
                sub[k] = dd[k][a:b]
            o = {k: (None if v is None else v[a:b]) for k, v in out.items()}
            solve(sub, o, stream=cr.cuda_stream)
            co.wait_stream(cr)
            with torch.cuda.stream(co):
                for k in outs:
                    hout[k][a:b].copy_(o[k], non_blocking=True)
        torch.cuda.synchronize()

    res = {}
    for chunks in chunk_counts:
        for k in outs:
            hout[k].zero_()
        one(chunks)                                         # warm-up
        t0 = time.perf_counter()
        for _ in range(steps):
            one(chunks)
        ms = (time.perf_counter() - t0) * 1e3 / steps
        res[chunks] = (ms, {k: v.numpy().copy() for k, v in hout.items()})
    in_b = sum(hin[k].numel() * hin[k].element_size() for k in per_inst)
    out_b = sum(hout[k].numel() * hout[k].element_size() for k in outs)
    return res, in_b, out_b


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c3")
    ap.add_argument("--mode", default=None,
                    help="search family: grid (every batch size), or '+'-joined greedy "
                         "(Alg. 2's greedy batching set), fixed-edge (no edge DVFS), binary "
                         "(whole-task offloading or local only), continuous (continuous CPU "
                         "frequency); default: the workload's own")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="instances the CPU oracle solves (default: about 15 s of work)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-e2e", action="store_true",
                    help="skip the host-resident (PCIe-inclusive) batches after the timed region")
    ap.add_argument("--no-stages", action="store_true",
                    help="skip timing the two-stage entry points after the timed region")
    ap.add_argument("--calibrate", action="store_true",
                    help="after the timed region, copy 1 GiB device-to-device 3 times "
                         "(reference dispatches for HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (got --gpus {args.gpus}); instances are "
              "independent, so several GPUs would each take a contiguous instance range "
              "through the same entry points", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2504_14611_amd import jdob
    from paper_2504_14611_amd import workloads as W

    w = W.WORKLOADS[args.workload]
    mode = w.mode if args.mode is None else parse_mode(args.mode)
    args.mode = mode_text(mode)
    cont = bool(mode & MODE_BITS["continuous"])
    grouped = w.name in GROUPED
    I, N, L, K, J = w.num_instances, w.N, w.L, w.K, w.J
    log(f"[bench] generating {w.name}: I={I} N={N} L={L} K={K} J={J} {w.dtype}")
    t0 = time.perf_counter()
    prob = W.generate(w)
    prob["mode"] = mode
    log(f"[bench] generated in {time.perf_counter() - t0:.1f}s; copying to the GPU")
    d = jdob.to_device(prob)
    if grouped:
        solve, alloc = jdob.solve_grouped, jdob.alloc_grouped
    else:
        solve, alloc = jdob.solve_batch, jdob.alloc_policy
    # one untimed launch that also fills the optional work counters (feasible
    # candidates and user evaluations, for the roofline); the timed launches
    # request only the policy
    counted = solve(d, alloc(d, counters=True))
    out = alloc(d, counters=False)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    for i in range(args.warmup):
        solve(d, out)
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} done")

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        solve(d, out)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms = [a.elapsed_time(b) for a, b in ev]
    ms_per_step = wall * 1e3 / args.steps
    kmean = float(np.mean(kern_ms))
    log(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step wall, kernel "
        f"mean {kmean:.3f} min {min(kern_ms):.3f} max {max(kern_ms):.3f} ms")

    host = jdob.to_host(out)
    hc = jdob.to_host(counted)
    keys = (("status", "num_groups", "energy", "group_end", "group_cut", "user_level") if grouped
            else ("status", "cut", "gpu_level", "batch", "energy", "user_level"))
    for k in keys:
        assert np.array_equal(host[k], hc[k], equal_nan=True), f"counting launch differs in {k}"
    F = int(hc["num_feasible"].astype(np.int64).sum())
    U = int(hc["num_user_evals"].sum())
    cand_per_inst = grouped_family_size(w, mode) if grouped else family_size(w, mode)
    cands = I * cand_per_inst
    ops = OPS_PER_CANDIDATE * F + model_ops_per_user_eval(w, mode) * U
    achieved = ops / (kmean * 1e-3)
    useful = USEFUL_PER_FEASIBLE_CAND * F + useful_ops_per_user_eval(w, mode) * U
    in_bytes, out_bytes = algorithmic_bytes(w, grouped, cont)

    tag = w.name if mode == w.mode else f"{w.name}_{args.mode.replace('+', '_')}"
    hetero = w.users is not None
    kfamily = (("jdob_hetero_grouped_kernel" if hetero else "jdob_grouped_kernel") if grouped else
               ("jdob_hetero_kernel" if hetero else "jdob_solve_kernel"))
    counters = measured_counters(kfamily, tag)
    T = "double" if w.dtype == "f64" else "float"
    one = "true" if (1 if mode & 2 else J) <= 64 else "false"
    ct = "true" if cont else "false"
    gr = "true" if mode & 1 else "false"
    if hetero:
        # without a continuous frequency the solve kernel is specialised to
        # the size of its level rows (4 <= 2^lg >= K)
        lg = max(2, int(np.ceil(np.log2(K)))) if not (cont or grouped) else 0
        kernel = (f"{kfamily}<{T},false,{gr},{ct},{lg}>" if not grouped else
                  f"{kfamily}<{T},false,{gr},{ct}>")
    elif grouped:
        kernel = (f"jdob_grouped_kernel<{T},false,false,true,{ct}>" if mode & 1 else
                  f"jdob_grouped_kernel<{T},{one},false,false,{ct}>")
    else:
        # queued evaluation of multi-level candidates from 17 users up (the
        # launch's own rule for the grid with CPU levels)
        qu = "true" if (w.N > 16 and not cont) else "false"
        kernel = (f"jdob_solve_kernel<{T},false,false,false,true,{ct},false>" if mode & 1 else
                  f"jdob_solve_kernel<{T},false,{one},false,false,{ct},{qu}>")
    res = {
        "metric": "candidate policies evaluated/sec + instances solved/sec on 1 MI355X",
        "value": cands / (ms_per_step * 1e-3),
        "unit": "candidates/s",
        "instances_per_s": I / (ms_per_step * 1e-3),
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "kernel_ms": kmean,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64" if w.dtype == "f64" else "f32", "data": "synthetic",
        "config": {"workload": f"{w.name}: {I} instances, N={N} users, L={L} layers, "
                               f"K={K} CPU levels, J={J} GPU levels"
                               + (", outer grouping" if grouped else "")
                               + (", heterogeneous users" if w.users is not None else ""),
                   "instances": I, "users": N, "layers": L, "cpu_levels": K, "gpu_levels": J,
                   "mode": args.mode, "entry": "jdob_solve_grouped" if grouped else "jdob_solve_batch",
                   "candidates_per_instance": cand_per_inst},
        "work": {"feasible_candidates": F, "user_evals": U,
                 "feasible_instances": int((host["status"] == 0).sum()),
                 "feasible_candidate_fraction": F / cands,
                 "user_evals_per_s": U / (kmean * 1e-3)},
        "roofline": {"bound": "alu", "achieved": achieved / 1e12, "peak": VALU_PEAK_OPS / 1e12,
                     "unit": "TOP/s", "frac": achieved / VALU_PEAK_OPS,
                     "traffic": counters.get("traffic"),
                     "valu_busy_counter": (counters.get("valu") or {}).get("busy"),
                     "valu_counters": counters.get("valu"),
                     "kernel": kernel,
                     "ops_per_launch": ops,
                     "ops_model": f"{OPS_PER_CANDIDATE} per feasible candidate + "
                                  f"{model_ops_per_user_eval(w, mode)} per offloader evaluation",
                     "useful_work": {"ops_per_launch": useful,
                                     "achieved": useful / (kmean * 1e-3) / 1e12,
                                     "frac": useful / (kmean * 1e-3) / VALU_PEAK_OPS,
                                     "model": f"{USEFUL_PER_FEASIBLE_CAND} per feasible candidate + "
                                              f"{useful_ops_per_user_eval(w, mode)} per offloader "
                                              "evaluation"},
                     "hbm_algorithmic_bytes": in_bytes + out_bytes,
                     "hbm_frac": (in_bytes + out_bytes) / (kmean * 1e-3) / HBM_PEAK},
        "cpu_baseline": None,
    }
    if grouped:
        res["work"]["inner_solves"] = int(hc["num_inner"].sum())
        res["work"]["groups_mean"] = float(host["num_groups"][host["status"] == 0].mean())
    res["roofline"]["source_sha256_16"] = source_hash()
    if not (args.no_stages or grouped or hetero):
        res["stages"] = time_stages(w, d, host, args.steps, args.warmup, stream)
        st = res["stages"]
        log(f"[bench] stage 1 {st['jdob_eval_user_tables']['ms']:.3f} ms "
            f"({st['jdob_eval_user_tables']['hbm_frac']:.3f} of HBM), "
            f"stage 2 {st['jdob_eval_joint']['ms']:.3f} ms")
    if not args.no_e2e:
        runs, in_b, out_b = end_to_end(prob, d, alloc, solve, E2E_STEPS, (1,) + E2E_PIECES)
        for chunks, (ms, hout) in runs.items():
            for k, v in hout.items():
                assert np.array_equal(v, host[k], equal_nan=True), \
                    f"end-to-end with {chunks} pieces differs in {k}"
            log(f"[bench] end-to-end, {chunks} piece(s): {ms:.3f} ms per batch")
        best = min(E2E_PIECES, key=lambda c: runs[c][0])

        def rate(ms):
            return {"ms": ms, "instances_per_s": I / (ms * 1e-3), "candidates_per_s": cands / (ms * 1e-3)}
        res["end_to_end"] = {
            "steps": E2E_STEPS, "host_memory": "pinned", "h2d_bytes": in_b, "d2h_bytes": out_b,
            "serial": dict(rate(runs[1][0]), chunks=1, streams=1),
            "pipelined": dict(rate(runs[best][0]), chunks=best, streams=3,
                              ms_by_chunks={str(c): runs[c][0] for c in E2E_PIECES})}
    if args.calibrate:
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] calibration copies: 3 x 1 GiB device-to-device")
        del src, dst
    if not args.no_cpu:
        sample = min(args.cpu_sample or CPU_SAMPLE.get(w.name, CPU_SAMPLE_DEFAULT), I)
        log(f"[bench] CPU oracle on {sample} instances (single thread)")
        o, cb = cpu_baseline(prob, w, sample, cand_per_inst, grouped)
        res["cpu_baseline"] = cb
        # spot parity of the timed run on the sample
        g = {k: (None if v is None else v[:sample]) for k, v in hc.items()}
        ps = {"instances": sample,
              "status_mismatch": int((g["status"] != o["status"]).sum()),
              "counter_mismatch": int(((g["num_feasible"] != o["num_feasible"])
                                       | (g["num_user_evals"] != o["num_user_evals"])).sum())}
        if grouped:
            ps["decision_mismatch"] = int(((g["num_groups"] != o["num_groups"])
                                           | (g["group_end"] != o["group_end"]).any(axis=1)
                                           | (g["group_cut"] != o["group_cut"]).any(axis=1)).sum())
        else:
            ps["decision_mismatch"] = int(((g["cut"] != o["cut"]) | (g["gpu_level"] != o["gpu_level"])
                                           | (g["batch"] != o["batch"])).sum())
        res["parity_sample"] = ps
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
