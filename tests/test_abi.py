"""The C-ABI library loads, exports what include/jdob.h declares, and rejects
invalid arguments on the host before any HIP call (so these run without a
GPU).  Every case below carries an argument error that validation must
catch; none of them can reach a kernel launch."""

import ctypes as C
import os
import re

import pytest

from paper_2504_14611_amd import jdob

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x1000  # never dereferenced: every call below fails validation first


def declared_functions():
    src = open(os.path.join(ROOT, "include", "jdob.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(jdob_[a-z_]+)\s*\(", src)))


def test_header_declares_the_documented_calls():
    assert declared_functions() == sorted(jdob.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = jdob.load()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings():
    lib = jdob.load()
    assert lib.jdob_status_string(0) == b"ok"
    assert lib.jdob_status_string(1) == b"invalid argument"
    assert lib.jdob_status_string(2) == b"unsupported size or dtype"
    assert lib.jdob_status_string(3) == b"HIP launch or device error"
    assert lib.jdob_status_string(-5) == b"unknown status"


def good_problem(**kw):
    p = jdob.Problem(16, 8, 6, 4, 4, jdob.JDOB_F32, *([FAKE] * 6), None, FAKE, FAKE,
                     1e-28, 0.5, 3.125e-26, 50.0)
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def good_policy(**kw):
    o = jdob.Policy(*([FAKE] * 8), None, None, None)
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def good_tables(**kw):
    t = jdob.UserTables(*([FAKE] * 8))
    for k, v in kw.items():
        setattr(t, k, v)
    return t


BAD_PROBLEMS = [
    ({"num_instances": -1}, jdob.JDOB_ERR_INVALID_ARG),
    ({"num_users": 0}, jdob.JDOB_ERR_INVALID_ARG),
    ({"num_layers": -1}, jdob.JDOB_ERR_INVALID_ARG),
    ({"num_local_levels": 0}, jdob.JDOB_ERR_INVALID_ARG),
    ({"num_gpu_levels": 0}, jdob.JDOB_ERR_INVALID_ARG),
    ({"num_users": 1025}, jdob.JDOB_ERR_UNSUPPORTED),
    ({"num_layers": 256}, jdob.JDOB_ERR_UNSUPPORTED),
    ({"num_local_levels": 65}, jdob.JDOB_ERR_UNSUPPORTED),
    ({"num_gpu_levels": 257}, jdob.JDOB_ERR_UNSUPPORTED),
    ({"dtype": 7}, jdob.JDOB_ERR_UNSUPPORTED),
    ({"layer_cycles": None}, jdob.JDOB_ERR_INVALID_ARG),
    ({"out_bits": None}, jdob.JDOB_ERR_INVALID_ARG),
    ({"gpu_alpha": None}, jdob.JDOB_ERR_INVALID_ARG),
    ({"gpu_beta": None}, jdob.JDOB_ERR_INVALID_ARG),
    ({"uplink_rate": None}, jdob.JDOB_ERR_INVALID_ARG),
    ({"deadline": None}, jdob.JDOB_ERR_INVALID_ARG),
    ({"local_freq": None}, jdob.JDOB_ERR_INVALID_ARG),
    ({"gpu_freq": None}, jdob.JDOB_ERR_INVALID_ARG),
    ({"kappa": float("nan")}, jdob.JDOB_ERR_INVALID_ARG),
    ({"p_tx": -1.0}, jdob.JDOB_ERR_INVALID_ARG),
    ({"gpu_c": float("inf")}, jdob.JDOB_ERR_INVALID_ARG),
    ({"gpu_p_static": -0.5}, jdob.JDOB_ERR_INVALID_ARG),
    ({"mode": 16}, jdob.JDOB_ERR_INVALID_ARG),
    ({"mode": -1}, jdob.JDOB_ERR_INVALID_ARG),
    ({"mode": jdob.JDOB_MODE_GREEDY | 16}, jdob.JDOB_ERR_INVALID_ARG),
    ({"mode": jdob.JDOB_MODE_CONTINUOUS_CPU | 32}, jdob.JDOB_ERR_INVALID_ARG),
    # per-instance LDS state above 64 KiB
    ({"num_users": 1024, "num_layers": 255, "num_local_levels": 64, "num_gpu_levels": 256,
      "dtype": jdob.JDOB_F64}, jdob.JDOB_ERR_UNSUPPORTED),
]


@pytest.mark.parametrize("fields,code", BAD_PROBLEMS)
def test_invalid_problem_rejected_by_every_entry_point(fields, code):
    lib = jdob.load()
    p = good_problem(**fields)
    pol, tab = good_policy(), good_tables()
    assert lib.jdob_solve_batch(C.byref(p), C.byref(pol), None) == code
    assert lib.jdob_eval_user_tables(C.byref(p), C.byref(tab), None) == code
    assert lib.jdob_eval_joint(C.byref(p), C.byref(tab), C.byref(pol), None) == code


ARRAYS = ("layer_cycles", "out_bits", "gpu_alpha", "gpu_beta", "uplink_rate", "deadline",
          "t_free", "local_freq", "gpu_freq")


def test_empty_batch_is_a_no_op_for_every_entry_point():
    """num_instances = 0: the other arguments are checked as usual, every
    array pointer may be NULL, nothing is launched (no HIP call is made, so
    this runs without a GPU) and the call succeeds."""
    lib = jdob.load()
    p = good_problem(num_instances=0, **{f: None for f in ARRAYS})
    pol = jdob.Policy(*([None] * len(jdob.Policy._fields_)))
    tab = jdob.UserTables(*([None] * len(jdob.UserTables._fields_)))
    grp = jdob.GroupedPolicy(*([None] * len(jdob.GroupedPolicy._fields_)))
    assert lib.jdob_solve_batch(C.byref(p), C.byref(pol), None) == jdob.JDOB_OK
    assert lib.jdob_eval_user_tables(C.byref(p), C.byref(tab), None) == jdob.JDOB_OK
    assert lib.jdob_eval_joint(C.byref(p), C.byref(tab), C.byref(pol), None) == jdob.JDOB_OK
    assert lib.jdob_solve_grouped(C.byref(p), C.byref(grp), None) == jdob.JDOB_OK
    # heterogeneous users: the solves accept an empty batch, the two stages
    # do not take such users at all
    p.user_zeta = FAKE
    assert lib.jdob_solve_batch(C.byref(p), C.byref(pol), None) == jdob.JDOB_OK
    assert lib.jdob_solve_grouped(C.byref(p), C.byref(grp), None) == jdob.JDOB_OK
    assert lib.jdob_eval_user_tables(C.byref(p), C.byref(tab), None) == jdob.JDOB_ERR_UNSUPPORTED
    # the rest is still checked
    for fields, code in (({"num_users": 0}, jdob.JDOB_ERR_INVALID_ARG),
                         ({"kappa": -1.0}, jdob.JDOB_ERR_INVALID_ARG),
                         ({"num_gpu_levels": 257}, jdob.JDOB_ERR_UNSUPPORTED),
                         ({"mode": 16}, jdob.JDOB_ERR_INVALID_ARG)):
        q = good_problem(num_instances=0, **{f: None for f in ARRAYS}, **fields)
        assert lib.jdob_solve_batch(C.byref(q), C.byref(pol), None) == code, fields
        assert lib.jdob_solve_grouped(C.byref(q), C.byref(grp), None) == code, fields


def test_rows_beyond_the_on_chip_budget_are_unsupported():
    """One instance's rows must fit 64 KB of LDS (see the header's limits):
    binary64 at N = 700 does not, and is refused before any launch."""
    lib = jdob.load()
    p = good_problem(num_users=700, num_layers=8, num_local_levels=16, num_gpu_levels=32,
                     dtype=jdob.JDOB_F64)
    assert lib.jdob_solve_batch(C.byref(p), C.byref(good_policy()), None) == jdob.JDOB_ERR_UNSUPPORTED
    assert lib.jdob_eval_joint(C.byref(p), C.byref(good_tables()), C.byref(good_policy()),
                               None) == jdob.JDOB_ERR_UNSUPPORTED


def test_mode_bits_match_the_header():
    src = open(os.path.join(ROOT, "include", "jdob.h")).read()
    for name, value in (("JDOB_MODE_GRID", jdob.JDOB_MODE_GRID),
                        ("JDOB_MODE_GREEDY", jdob.JDOB_MODE_GREEDY),
                        ("JDOB_MODE_FIXED_EDGE_FREQ", jdob.JDOB_MODE_FIXED_EDGE_FREQ),
                        ("JDOB_MODE_BINARY", jdob.JDOB_MODE_BINARY),
                        ("JDOB_MODE_CONTINUOUS_CPU", jdob.JDOB_MODE_CONTINUOUS_CPU)):
        assert re.search(rf"\b{name} = {value}\b", src), name


def test_problem_struct_layout():
    # the binding's struct must match the header's field order and padding
    assert jdob.Problem.mode.offset == 6 * 4 + 9 * 8 + 4 * 8
    assert jdob.Problem.user_zeta.offset == jdob.Problem.mode.offset + 8
    assert C.sizeof(jdob.Problem) == jdob.Problem.user_local_freq.offset + 8


def good_grouped(**kw):
    g = jdob.GroupedPolicy(*([FAKE] * 14), None, None, None, None)
    for k, v in kw.items():
        setattr(g, k, v)
    return g


@pytest.mark.parametrize("fields,code", BAD_PROBLEMS + [({"num_users": 65}, jdob.JDOB_ERR_UNSUPPORTED)])
def test_invalid_problem_rejected_by_grouped(fields, code):
    lib = jdob.load()
    p = good_problem(**fields)
    assert lib.jdob_solve_grouped(C.byref(p), C.byref(good_grouped()), None) == code


@pytest.mark.parametrize("field", [f for f, _ in jdob.GroupedPolicy._fields_
                                   if f not in ("num_inner", "num_feasible", "num_user_evals",
                                                "user_freq")])
def test_missing_grouped_output_rejected(field):
    lib = jdob.load()
    p = good_problem()
    g = good_grouped(**{field: None})
    assert lib.jdob_solve_grouped(C.byref(p), C.byref(g), None) == jdob.JDOB_ERR_INVALID_ARG
    assert lib.jdob_solve_grouped(C.byref(p), None, None) == jdob.JDOB_ERR_INVALID_ARG


def test_null_structs_rejected():
    lib = jdob.load()
    assert lib.jdob_solve_batch(None, None, None) == jdob.JDOB_ERR_INVALID_ARG
    p = good_problem(num_users=0)
    assert lib.jdob_solve_batch(C.byref(p), None, None) == jdob.JDOB_ERR_INVALID_ARG


@pytest.mark.parametrize("field", [f for f, _ in jdob.Policy._fields_
                                   if f not in ("num_feasible", "num_user_evals", "user_freq")])
def test_missing_policy_output_rejected(field):
    lib = jdob.load()
    p, tab = good_problem(), good_tables()
    pol = good_policy(**{field: None})
    assert lib.jdob_solve_batch(C.byref(p), C.byref(pol), None) == jdob.JDOB_ERR_INVALID_ARG
    assert lib.jdob_eval_joint(C.byref(p), C.byref(tab), C.byref(pol), None) == \
        jdob.JDOB_ERR_INVALID_ARG
    assert lib.jdob_solve_batch(C.byref(p), None, None) == jdob.JDOB_ERR_INVALID_ARG


@pytest.mark.parametrize("field", [f for f, _ in jdob.UserTables._fields_])
def test_missing_table_rejected(field):
    lib = jdob.load()
    p, pol = good_problem(), good_policy()
    tab = good_tables(**{field: None})
    assert lib.jdob_eval_user_tables(C.byref(p), C.byref(tab), None) == jdob.JDOB_ERR_INVALID_ARG
    assert lib.jdob_eval_joint(C.byref(p), C.byref(tab), C.byref(pol), None) == \
        jdob.JDOB_ERR_INVALID_ARG


def test_binding_fails_loudly_without_library(tmp_path):
    saved = jdob._lib
    jdob._lib = None
    try:
        with pytest.raises(OSError):
            jdob.load(str(tmp_path / "missing.so"))
    finally:
        jdob._lib = saved


def _header_fields(struct_name):
    """Field names of a typedef'd struct in include/jdob.h, in order."""
    src = open(os.path.join(ROOT, "include", "jdob.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    body = re.search(r"typedef struct \{([^}]*)\}\s*" + struct_name + r";", src).group(1)
    return [re.search(r"(\w+)\s*;", d + ";").group(1) for d in body.split(";") if d.strip()]


@pytest.mark.parametrize("struct,cls", [("jdob_problem", jdob.Problem), ("jdob_policy", jdob.Policy),
                                        ("jdob_user_tables", jdob.UserTables),
                                        ("jdob_grouped_policy", jdob.GroupedPolicy)])
def test_binding_structs_follow_the_header(struct, cls):
    assert [k for k, _ in cls._fields_] == _header_fields(struct)


@pytest.mark.parametrize("fields,code", BAD_PROBLEMS)
def test_invalid_heterogeneous_problem_rejected(fields, code):
    lib = jdob.load()
    p = good_problem(user_zeta=FAKE, **fields)
    assert lib.jdob_solve_batch(C.byref(p), C.byref(good_policy()), None) == code


@pytest.mark.parametrize("field", ["user_zeta", "user_kappa", "user_p_tx", "user_local_freq"])
def test_heterogeneous_users_not_through_the_two_stages(field):
    lib = jdob.load()
    p = good_problem(**{field: FAKE})
    pol, tab = good_policy(), good_tables()
    assert lib.jdob_eval_user_tables(C.byref(p), C.byref(tab), None) == jdob.JDOB_ERR_UNSUPPORTED
    assert lib.jdob_eval_joint(C.byref(p), C.byref(tab), C.byref(pol), None) == \
        jdob.JDOB_ERR_UNSUPPORTED
    # limits of the heterogeneous kernels (checked before any launch): 64
    # users, and their LDS
    g = good_grouped()
    q = good_problem(num_users=65, **{field: FAKE})
    assert lib.jdob_solve_batch(C.byref(q), C.byref(pol), None) == jdob.JDOB_ERR_UNSUPPORTED
    assert lib.jdob_solve_grouped(C.byref(q), C.byref(g), None) == jdob.JDOB_ERR_UNSUPPORTED
    q = good_problem(num_users=64, num_layers=255, num_local_levels=64, num_gpu_levels=256,
                     dtype=jdob.JDOB_F64, **{field: FAKE})
    assert lib.jdob_solve_batch(C.byref(q), C.byref(pol), None) == jdob.JDOB_ERR_UNSUPPORTED
    assert lib.jdob_solve_batch(C.byref(q), None, None) == jdob.JDOB_ERR_UNSUPPORTED
    assert lib.jdob_solve_grouped(C.byref(q), C.byref(g), None) == jdob.JDOB_ERR_UNSUPPORTED
    # a missing grouped output is rejected before any launch
    q = good_problem(**{field: FAKE})
    assert lib.jdob_solve_grouped(C.byref(q), C.byref(good_grouped(order=None)), None) == \
        jdob.JDOB_ERR_INVALID_ARG


def _table_formula_bytes(I, N, L, szP):
    """Evaluate the stage-1 output size written in the comment above
    jdob_eval_user_tables."""
    src = open(os.path.join(ROOT, "include", "jdob.h")).read()
    m = re.search(r"Output size:\s*([^\n]*?)\s*bytes", src)
    assert m, "the header states the stage-1 output size"
    expr = m.group(1).replace("sizeof(P)", "szP")
    assert re.fullmatch(r"[ILN0-9szP+*() ]+", expr), expr
    return eval(expr, {}, {"I": I, "N": N, "L": L, "szP": szP})


def _table_struct_bytes(I, N, L, szP):
    """Bytes of the jdob_user_tables fields from their declared types and the
    [..] extents of their comments."""
    src = open(os.path.join(ROOT, "include", "jdob.h")).read()
    body = re.findall(r"typedef struct \{((?:(?!typedef).)*?)\} jdob_user_tables;", src, flags=re.S)[0]
    size = {"int16_t": 2, "int32_t": 4, "int8_t": 1, "void": szP}
    total, fields = 0, 0
    for typ, name, dims in re.findall(r"(int16_t|int32_t|int8_t|void)\s*\*(\w+);\s*/\*\s*((?:\[[^\]]+\])+)",
                                      body):
        n = 1
        for d in re.findall(r"\[([^\]]+)\]", dims):
            n *= eval(d, {}, {"I": I, "N": N, "L": L})
        total += n * size[typ]
        fields += 1
    assert fields == len(jdob.UserTables._fields_)
    return total


@pytest.mark.parametrize("I,N,L,dtype", [(1, 1, 1, "f32"), (3, 32, 22, "f32"), (5, 128, 50, "f32"),
                                         (2, 7, 9, "f64"), (4, 1024, 3, "f64")])
def test_stage1_output_size_in_header_matches_the_tables(I, N, L, dtype):
    """The size a caller would allocate from the header equals the bytes the
    binding allocates and the fields the struct declares."""
    import torch
    szP = 8 if dtype == "f64" else 4
    d = {"rate": torch.empty((I, N)), "N": N, "L": L, "dtype": dtype}
    alloc = sum(t.numel() * t.element_size() for t in jdob.alloc_tables(d).values())
    assert _table_formula_bytes(I, N, L, szP) == alloc
    assert _table_struct_bytes(I, N, L, szP) == alloc
