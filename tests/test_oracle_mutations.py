"""Planted mistakes in a copy of the oracle must be caught by its pins.

Each mutation edits one line of a temporary copy of the oracle source (a
dropped term, a wrong index, a transposed operand, a reversed order), builds
it with the same flags, and runs a short battery of the pins of
test_oracle*.py: closed
forms, the exact-rational enumerations and the brute force.  The real
oracle is restored afterwards.
"""

import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from paper_2504_14611_amd import workloads as W
from tests import exact_model
from tests.test_oracle import one_user, tiny
from tests.test_oracle_grouped import og_tiny

HETERO = "jdob_oracle_hetero.h"

MUTATIONS = {
    "drop_upload_energy": ("acc = acc + (e + ptx * w->up[i * (L + 1) + s]);", "acc = acc + (e);"),
    "batch_deadline_off_by_one": ("REAL H = w->lo[b] - Phi;", "REAL H = w->lo[b > 1 ? b - 1 : 1] - Phi;"),
    "batch_size_off_by_one": ("REAL Phi = (w->A[s] + w->B[s] * (REAL)b) * w->r[j];",
                              "REAL Phi = (w->A[s] + w->B[s] * (REAL)(b - 1)) * w->r[j];"),
    "rate_order_reversed": ("while (c >= 0 && (rate[w->pi[c]] < rate[x] ||",
                            "while (c >= 0 && (rate[w->pi[c]] > rate[x] ||"),
    "gpu_stretch_transposed": ("w->r[j] = g[J - 1] / g[j];", "w->r[j] = g[j] / g[J - 1];"),
    "local_energy_linear_in_f": ("REAL eps = kappa * (f[k] * f[k]);", "REAL eps = kappa * f[k];"),
    "release_without_batch": ("return ready + Phi;", "return ready;"),
    "gpu_free_time_ignored": ("if (!(H >= w->tfree)) return 0;", "if (!(H >= 0)) return 0;"),
    "suffix_sum_skips_layer": ("w->A[s] = w->A[s + 1] + al[s];", "w->A[s] = w->A[s + 1] + (s > 0 ? al[s] : 0);"),
    # the search variants
    "greedy_threshold_of_fastest_user": ("return w->t[s * K + K - 1] <= slack - w->up[(b - 1) * (L + 1) + s];",
                                         "return w->t[s * K + K - 1] <= slack - w->up[s];"),
    "greedy_threshold_at_top_level": ("while (b >= 1 && !FN(meets_threshold)(w, s, j, b)) --b;",
                                      "while (b >= 1 && !FN(meets_threshold)(w, s, J - 1, b)) --b;"),
    "greedy_keeps_whole_list": ("while (b >= 1 && !FN(meets_threshold)(w, s, j, b)) --b;",
                                "while (0) --b;"),
    "greedy_drops_one_more": ("if (b == 0) break;", "if (b == 0) break; if (b > 1) --b;"),
    "binary_keeps_every_cut": ("(p->mode & JO_MODE_BINARY) ? 1 : L", "(p->mode & JO_MODE_BINARY) ? L : L"),
    "fixed_edge_ignored": ("(p->mode & JO_MODE_FIXED_EDGE) ? J - 1 : 0", "(p->mode & JO_MODE_FIXED_EDGE) ? 0 : 0"),
    # continuous CPU frequency
    "continuous_without_lower_clamp": ("return g < w->fmin ? w->fmin : (g > w->fmax ? w->fmax : g);",
                                       "return g > w->fmax ? w->fmax : g;"),
    "continuous_release_at_top_frequency": ("REAL tl = w->cont ? w->C[s] / w->fz[i] : w->t[s * K + w->lv[i]];",
                                            "REAL tl = w->cont ? w->C[s] / w->fmax : w->t[s * K + w->lv[i]];"),
    "continuous_local_at_top_frequency": ("w->fL[m] = FN(cont_freq)(w, w->C[L], T[m]);",
                                          "w->fL[m] = w->fmax;"),
    # outer grouping
    "grouping_release_not_chained": ("FN(group_problem)(p, inst, ord, j, i, &fT[j * F + k], grate, gdl, gid, gu, &sub);\n"
                                     "          JO_CAT(jo_best, SFX) r = FN(group_solve)(&sub, &w, &hw);",
                                     "FN(group_problem)(p, inst, ord, j, i, &fT[0], grate, gdl, gid, gu, &sub);\n"
                                     "          JO_CAT(jo_best, SFX) r = FN(group_solve)(&sub, &w, &hw);"),
    "grouping_winner_shared_without_test": ("            if (!FN(group_eval)(&sub, &w, &hw, r.s, r.j, r.b, &E, &tf)) break;",
                                            "            FN(group_eval)(&sub, &w, &hw, r.s, r.j, r.b, &E, &tf);"),
    "grouping_by_deadline_descending": ("while (c >= 0 && (T[ord[c]] > T[x] || (T[ord[c]] == T[x] && ord[c] > x))) {",
                                        "while (c >= 0 && (T[ord[c]] < T[x] || (T[ord[c]] == T[x] && ord[c] > x))) {"),
    "grouping_keeps_first_feasible": ("    if (fE[q] <= E && fT[q] <= T) return;", "    if (q >= 0) return;"),
    "grouping_single_users_only": ("for (int j = 0; j < i; ++j) { /* last group: ord[j..i-1] */",
                                   "for (int j = i - 1; j < i; ++j) { /* last group: ord[j..i-1] */"),
    "grouping_one_state_per_prefix": ("  *n = m + 1 < JO_FRONT ? m + 1 : JO_FRONT;\n}", "  *n = 1;\n}"),
    "grouping_dominance_by_energy_only": ("if (!(E <= fE[q] && T <= fT[q])) {", "if (!(E <= fE[q])) {"),
    # stage-1 tables (jo_user_tables)
    "tables_gamma_at_lowest_level": ("out->gamma[o] = up + w.t[s * K + K - 1];",
                                     "out->gamma[o] = up + w.t[s * K];"),
    "tables_energy_without_upload": ("out->self_energy[o] = (k >= 0) ? w.e[s * K + k] + ptx * up : (REAL)INFINITY;",
                                     "out->self_energy[o] = (k >= 0) ? w.e[s * K + k] : (REAL)INFINITY;"),
    "tables_slack_at_top_level": ("out->self_slack[o] = budget - w.t[s * K + (k >= 0 ? k : K - 1)];",
                                  "out->self_slack[o] = budget - w.t[s * K + K - 1];"),
    "tables_rate_by_position": ("REAL up = (s < L) ? bits[s] / rate[m] : (REAL)0;",
                                "REAL up = (s < L) ? bits[s] / rate[w.pi[m]] : (REAL)0;"),
    "tables_row_L_uploads": ("REAL up = (s < L) ? bits[s] / rate[m] : (REAL)0;",
                             "REAL up = bits[s] / rate[m];"),
    "tables_level_against_deadline_alone": ("int k = FN(lowest_level)(w.t + s * K, K, budget);",
                                            "int k = FN(lowest_level)(w.t + s * K, K, T[m]);"),
    "tables_highest_fitting_level": ("int k = FN(lowest_level)(w.t + s * K, K, budget);",
                                     "int k = FN(lowest_level)(w.t + s * K, K, budget); "
                                     "while (k >= 0 && k + 1 < K && w.t[s * K + k + 1] <= budget) ++k;"),
    # heterogeneous users (jdob_oracle_hetero.h)
    "hetero_zeta_in_energy": (HETERO, "HE(w, m, s, k) = (w->kap[m] * (fk * fk)) * w->C[s];",
                              "HE(w, m, s, k) = (w->kap[m] * (fk * fk)) * W;"),
    "hetero_zeta_ignored": (HETERO, "HT(w, m, s, k) = W / fk;", "HT(w, m, s, k) = w->C[s] / fk;"),
    "hetero_shared_kappa": (HETERO, "w->kap[m] = p->user_kappa ? p->user_kappa[o] : (REAL)p->kappa;",
                            "w->kap[m] = (REAL)p->kappa;"),
    "hetero_power_by_position": (HETERO, "acc = acc + (e + w->ptx[m] * HU(w, m, s));",
                                 "acc = acc + (e + w->ptx[i] * HU(w, m, s));"),
    "hetero_shared_levels": (HETERO, "w->f[m * K + k] = p->user_local_freq ? p->user_local_freq[o * K + k] : p->local_freq[k];",
                             "w->f[m * K + k] = p->local_freq[k];"),
    "hetero_order_by_upload_only": (HETERO, "const REAL gx = HU(w, x, s) + HT(w, x, s, K - 1);",
                                    "const REAL gx = HU(w, x, s);"),
    "hetero_greedy_tests_fastest_only": (HETERO, "if (!(HT(w, m, s, K - 1) <= H - HU(w, m, s))) return 0;",
                                         "if (i == 0 && !(HT(w, m, s, K - 1) <= H - HU(w, m, s))) return 0;"),
    "hetero_continuous_range_of_user_0": (HETERO, "const REAL lo = w->f[m * w->K], hi = w->f[m * w->K + w->K - 1];",
                                          "const REAL lo = w->f[0], hi = w->f[w->K - 1];"),
    "hetero_group_parameters_by_position": ("const size_t o = (size_t)inst * N + gid[q];",
                                            "const size_t o = (size_t)inst * N + q;"),
}


def _build_mutant(tmp, name):
    src = os.path.dirname(oracle.__file__)
    d = tmp / name
    d.mkdir()
    for f in oracle._SOURCES + oracle._HEADERS:
        shutil.copy(os.path.join(src, f), d / f)
    m = MUTATIONS[name]
    target, old, new = m if len(m) == 3 else ("jdob_oracle_body.h", *m)
    body = (d / target).read_text()
    assert body.count(old) == 1, name
    (d / target).write_text(body.replace(old, new))
    so = d / "lib.so"
    subprocess.run(["gcc", *oracle.CFLAGS, "-o", str(so), str(d / "jdob_oracle.c"),
                    str(d / "jdob_brute.c"), "-lm"], check=True)
    lib = ctypes.CDLL(str(so))
    oracle._declare(lib)
    return lib


class _Caught(Exception):
    """A pin failed and the battery stops there."""


def _pins_fail(stop=False):
    """Names of the pins that fail with the currently loaded oracle; with
    stop, only the first (a planted mistake needs one failing pin)."""
    failed = []

    def fail(label):
        failed.append(label)
        if stop:
            raise _Caught()

    try:
        _battery(fail, failed)
    except _Caught:
        pass
    return failed


def _battery(fail, failed):
    _tables_pins_fail(fail)  # the cheapest first
    _hetero_hand_fail(fail)
    o = oracle.solve(one_user(0.6))
    if not (o["energy"][0] == pytest.approx(0.2125, rel=1e-15)
            and o["t_free_out"][0] == pytest.approx(0.102, rel=1e-15)):
        fail("closed_form")
    o = oracle.solve(one_user(0.45, t_free=0.449))
    if o["status"][0] != 1:
        fail("closed_form_busy_gpu")
    p = W.generate(W.WORKLOADS["c0"], 0, 48)
    o = oracle.solve(p)
    for inst in range(48):
        bf = oracle.brute(p, inst, suffix_only=False)
        if bf["found"] != (o["status"][inst] == 0) or (
                bf["found"] and not o["energy"][inst] == pytest.approx(bf["energy"], rel=1e-12)):
            fail("brute_force_c0")
            break
    p = tiny(4, 4, 3, 3, 32, deadline=("per_user", 0.03, 0.4), stream=341)
    o = oracle.solve(p)
    for inst in range(32):
        bf = oracle.brute(p, inst, suffix_only=True)
        if bf["found"] != (o["status"][inst] == 0) or (
                bf["found"] and not o["energy"][inst] == pytest.approx(bf["energy"], rel=1e-12)):
            fail("brute_force_per_user_deadlines")
            break
    p = tiny(3, 3, 2, 3, 6, deadline=("per_user", 0.05, 0.5), stream=77)
    o = oracle.solve(p)
    for inst in range(6):
        ex = exact_model.solve_exact(p, inst, suffix_only=True)
        if (ex is None) != (o["status"][inst] == 1) or (ex is not None and not (
                o["energy"][inst] == pytest.approx(float(ex["energy"]), rel=1e-13)
                and o["t_free_out"][inst] == pytest.approx(float(ex["t_free_out"]), rel=1e-13))):
            fail("exact_rational")
            break
    # per-user deadlines over a wide range: partial greedy batches win on
    # about one instance in eight
    p = tiny(4, 3, 3, 4, 64, deadline=("per_user", 0.02, 0.8), stream=740)
    for mode, label, n in ((oracle.MODE_GREEDY, "exact_greedy", 64),
                           (oracle.MODE_FIXED_EDGE, "exact_fixed_edge", 14),
                           (oracle.MODE_BINARY, "exact_binary", 14)):
        q = dict(p)
        q["mode"] = mode
        o = oracle.solve(q)
        for inst in range(n):
            ex = exact_model.solve_exact(q, inst, suffix_only=True)
            if (ex is None) != (o["status"][inst] == 1) or (ex is not None and not (
                    o["energy"][inst] == pytest.approx(float(ex["energy"]), rel=1e-13)
                    and o["batch"][inst] == ex["batch"])):
                fail(label)
                break
    p = tiny(4, 4, 3, 3, 12, deadline=("per_user", 0.03, 0.4), stream=860)
    p["mode"] = oracle.MODE_CONTINUOUS
    o = oracle.solve(p)
    for inst in range(12):
        ex = exact_model.solve_exact(p, inst, suffix_only=True)
        if (ex is None) != (o["status"][inst] == 1) or (ex is not None and not (
                o["energy"][inst] == pytest.approx(float(ex["energy"]), rel=1e-12)
                and o["t_free_out"][inst] == pytest.approx(float(ex["t_free_out"]), rel=1e-12))):
            fail("exact_continuous")
            break
    for shape, stream in (((3, 3, 2, 3), 810), ((4, 3, 3, 2), 811)):
        p = og_tiny(*shape, 10, stream)
        o = oracle.solve_grouped(p)
        for inst in range(10):
            ex = exact_model.solve_grouped_exact(p, inst)
            if (ex is None) != (o["status"][inst] == 1) or (ex is not None and not (
                    o["energy"][inst] == pytest.approx(float(ex["energy"]), rel=1e-12)
                    and o["t_free_out"][inst] == pytest.approx(float(ex["t_free_out"]), rel=1e-12))):
                fail("exact_grouping")
                break
        if "exact_grouping" in failed:
            break
    from tests.test_oracle_grouped import brute_force_grouping
    p = W.generate(W.WORKLOADS["p5"].replace(N=6, num_instances=8, stream=833))
    o = oracle.solve_grouped(p)
    for inst in range(8):
        if not o["energy"][inst] == pytest.approx(brute_force_grouping(p, inst), rel=1e-6):
            fail("grouping_brute_force")
            break
    _hetero_pins_fail(fail)


def _tables_pins_fail(fail):
    """The pins of test_oracle_tables.py, one short case each."""
    from tests import test_oracle_tables as TT
    if TT.hand_case_mismatches("f64"):
        fail("tables_by_hand")
    bad, _ = TT.exact_mismatches(tiny(5, 4, 3, 2, 8, deadline=("per_user", 0.01, 0.6), stream=901), 8)
    if bad:
        fail("tables_exact")


def _hetero_hand_fail(fail):
    """The two-user case of test_oracle_hetero.py worked by hand."""
    from tests import test_oracle_hetero as H
    p = H.two_users()
    o = oracle.solve(p)
    c = oracle.eval_candidate(p, 0, 1, 0, 1)
    if not (o["energy"][0] == pytest.approx(0.6875, rel=1e-15)
            and c["energy"] == pytest.approx(2.1725, rel=1e-15)
            and list(c["user_offload"]) == [0, 1]):
        fail("hetero_by_hand")


def _hetero_pins_fail(fail):
    """The other pins of test_oracle_hetero.py, one short case each."""
    from tests import test_oracle_hetero as H
    p = H.htiny(4, 3, 3, 3, 24, 1201)
    o = oracle.solve(p)
    for inst in range(24):
        bf = oracle.brute(p, inst, suffix_only=True)
        if bf["found"] != (o["status"][inst] == 0) or (
                bf["found"] and not o["energy"][inst] == pytest.approx(bf["energy"], rel=1e-12)):
            fail("hetero_brute_force")
            break
    for mode in (oracle.MODE_GREEDY, oracle.MODE_CONTINUOUS):
        p = H.with_mode(H.htiny(4, 4, 3, 3, 16, 1211), mode)
        o = oracle.solve(p)
        for inst in range(16):
            ex = exact_model.solve_exact(p, inst, suffix_only=True)
            if (ex is None) != (o["status"][inst] == 1) or (ex is not None and not (
                    o["energy"][inst] == pytest.approx(float(ex["energy"]), rel=1e-12))):
                fail(f"hetero_exact_{mode}")
                break
    p = H.og_htiny(4, 3, 3, 2, 10, 1241)
    o = oracle.solve_grouped(p)
    for inst in range(10):
        ex = exact_model.solve_grouped_exact(p, inst)
        if (ex is None) != (o["status"][inst] == 1) or (ex is not None and not (
                o["energy"][inst] == pytest.approx(float(ex["energy"]), rel=1e-12))):
            fail("hetero_exact_grouping")
            break
    p = W.generate(W.WORKLOADS["h2"], 0, 256)
    q, cs = H._rescaled(p, 3)
    a, b = oracle.solve(p), oracle.solve(q)
    if not (np.array_equal(a["energy"], b["energy"]) and np.array_equal(a["cut"], b["cut"])):
        fail("hetero_rescaling")


def test_pins_pass_on_the_real_oracle():
    assert _pins_fail() == []


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(tmp_path, name):
    real = oracle.lib()
    try:
        oracle._lib = _build_mutant(tmp_path, name)
        failed = _pins_fail(stop=True)
    finally:
        oracle._lib = real
    assert failed, f"mutation {name} went unnoticed"
