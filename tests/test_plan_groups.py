"""Host-side checks of the XOR-group and Ring plans of libar.so (no GPU).

The group of Table 1b (t_k(x) = x XOR k, power-of-two P) gives Recursive
Halving, Recursive Doubling and their hybrid (Secs. 7-9, closing remarks);
the Ring is Sec. 6.  Each plan's launch tables run through the numpy
interpreter of test_plan_host (forward, reversed and from a snapshot) and
must reproduce the oracle's bits; the plan's sizes must equal the oracle's
counts of the same schedule.
"""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2004_09362_amd import ar
from test_plan_host import interpret

POW2 = [1, 2, 4, 8, 16, 32, 64, 128]


def ceil_log2(P):
    return max(0, (P - 1).bit_length())


def ks(P):
    L = ceil_log2(P)
    return list(range(L, 2 * L + 1))


def cases():
    out = [(P, k, "xor", "butterfly") for P in POW2 for k in ks(P)]
    out += [(P, 2 * (P - 1), "cyclic", "ring") for P in list(range(1, 20)) + [31, 37, 64, 127, 128]]
    return out


@pytest.mark.parametrize("P,k,group,schedule", cases())
def test_sizes_match_oracle_counts(P, k, group, schedule):
    plan = ar.Plan(P, 10 * P + 3, "float32", "sum", k, group=group, schedule=schedule)
    st = plan.stats()
    assert (st.group, st.schedule) == (ar._group_code(group), ar._schedule_code(schedule))
    assert st.fused_ok == int(P >= 2)
    if P <= 9 or schedule != "ring":   # the oracle's trace holds 16 steps
        t = oracle.Terms(P, k, group=group, schedule=schedule)
        tr = t.trace
        assert (st.rs_steps, st.ag_steps) == (tr.rs_steps, tr.ag_steps)
        assert st.blocks_pulled_per_rank == sum(tr.pulls[:k])
        assert st.combines_per_rank == sum(tr.combines[:tr.rs_steps])
        launches = [l for l in plan.launches() if l[0] != 2]
        assert len(launches) == k
        for s, (phase, ranges) in enumerate(launches):
            if group == "xor":
                pulled = {(r["src"], (r["p0"] + j) ^ r["delta"]) for r in ranges if r["delta"] != 0
                          for j in range(r["count"])}
            else:
                pulled = {(r["src"], (r["p0"] + j + r["delta"]) % P) for r in ranges if r["delta"] != 0
                          for j in range(r["count"])}
            assert len(pulled) == tr.pulls[s], (P, k, s)
    assert st.bytes_pulled_total == st.blocks_pulled_per_rank * st.n * 4
    if schedule == "ring":
        assert (st.rs_steps, st.ag_steps, st.launches) == (P - 1, P - 1, 2 * (P - 1))
        assert st.blocks_pulled_per_rank == 2 * (P - 1) and st.combines_per_rank == P - 1
    if schedule == "ring" or k == 2 * ceil_log2(P):
        # Ring and Recursive Halving: in place, 5 (P-1) blocks of HBM traffic per rank
        assert st.hbm_bytes_stepwise == 5 * (P - 1) * st.n * 4
        assert st.workspace_bytes == 0
        for phase, ranges in plan.launches():
            for r in ranges:
                assert r["dst"] == 0 and r["src"] == 0 and r["own"] in (0, -1)
    if group == "xor":
        assert st.launches == k + (1 if (P == 2 and k == 1) else 0)


@pytest.mark.parametrize("P,k,group,schedule", [c for c in cases() if c[0] <= 32 or c[3] == "ring" and c[0] <= 37])
def test_tables_reproduce_oracle_bits(P, k, group, schedule):
    rng = np.random.default_rng(2000 + P + 7 * k)
    for n in (2 * P + 5, max(P - 1, 1)):
        plan = ar.Plan(P, n, "float32", "sum", k, group=group, schedule=schedule)
        x = (rng.normal(size=(P, n)) * np.exp2(rng.integers(-8, 8, size=(P, n)))).astype(np.float32)
        want = oracle.allreduce(x, k, "sum", group=group, schedule=schedule)
        for order in ("forward", "reverse", "snapshot"):
            got = interpret(plan, x, "sum", order)
            assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), (P, k, n, order)


@pytest.mark.parametrize("P,k,group,schedule", [(8, 3, "xor", "butterfly"), (8, 4, "xor", "butterfly"),
                                                (16, 7, "xor", "butterfly"), (5, 8, "cyclic", "ring"),
                                                (12, 22, "cyclic", "ring")])
def test_tables_int32_and_max(P, k, group, schedule):
    rng = np.random.default_rng(P + k)
    n = 3 * P + 2
    xi = rng.integers(-2**31, 2**31, size=(P, n), dtype=np.int64).astype(np.int32)
    xf = rng.normal(size=(P, n)).astype(np.float32)
    xf[0, :3] = -0.0
    for arr, dt, op in ((xi, "int32", "sum"), (xi, "int32", "max"), (xf, "float32", "max")):
        plan = ar.Plan(P, n, dt, op, k, group=group, schedule=schedule)
        got = interpret(plan, arr, op)
        want = oracle.allreduce(arr, k, op, group=group, schedule=schedule)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), (op, dt)


@pytest.mark.parametrize("args", [
    (6, 10, 1, 0, 3, ar.AR_GROUP_XOR, ar.AR_SCHEDULE_BUTTERFLY),     # not a power of two
    (8, 10, 1, 0, 2, ar.AR_GROUP_XOR, ar.AR_SCHEDULE_BUTTERFLY),     # k outside [L, 2L]
    (8, 10, 1, 0, 14, ar.AR_GROUP_XOR, ar.AR_SCHEDULE_RING),         # the Ring is cyclic
    (7, 10, 1, 0, 6, ar.AR_GROUP_CYCLIC, ar.AR_SCHEDULE_RING),       # Ring needs k = 2(P-1)
    (7, 10, 1, 0, 6, 2, ar.AR_SCHEDULE_BUTTERFLY),                   # unknown group
    (7, 10, 1, 0, 6, ar.AR_GROUP_CYCLIC, 5),                         # unknown schedule
])
def test_create_ex_rejects(args):
    h = ctypes.c_void_p()
    assert ar.lib.ar_plan_create_ex(*args, ctypes.byref(h)) == ar.AR_ERR_INVALID_ARG
    assert h.value is None
    assert ar.ar_last_error() != ""


def test_create_ex_rejects_P_above_the_compiled_maximum():
    h = ctypes.c_void_p()
    args = (129, 10, 1, 0, 256, ar.AR_GROUP_CYCLIC, ar.AR_SCHEDULE_RING)
    assert ar.lib.ar_plan_create_ex(*args, ctypes.byref(h)) == ar.AR_ERR_UNSUPPORTED
    assert h.value is None and "128" in ar.ar_last_error()


def test_create_ex_defaults_equal_create():
    for P in (5, 8, 37):
        for k in ks(P):
            a = ar.Plan(P, 100, "float32", "sum", k).launches()
            h = ar.ar_plan_create(P, 100, "float32", "sum", k)
            try:
                b = [ar.ar_plan_launch(h, i) for i in range(ar.ar_plan_num_launches(h))]
            finally:
                ar.ar_plan_destroy(h)
            assert a == b


def test_xor_hybrid_costs_no_more_than_cyclic():
    """For power-of-two P the XOR group's shifted schedules coincide while
    f_i >= w, so its hybrid never receives more blocks than the cyclic
    group's Sec. 8 schedule, and strictly fewer for 0 < r < L (P >= 8)."""
    for P in (8, 16, 32, 64, 128):
        L = ceil_log2(P)
        for k in ks(P):
            x = ar.Plan(P, 1000, "float32", "sum", k, group="xor").stats().blocks_pulled_per_rank
            c = ar.Plan(P, 1000, "float32", "sum", k).stats().blocks_pulled_per_rank
            r = 2 * L - k
            assert x <= c
            if 0 < r < L:
                assert x < c, (P, k)


# ---------------------------------------------------------------------------
# Randomised: any group, schedule, P, k and ragged n
# ---------------------------------------------------------------------------

from hypothesis import HealthCheck, given, settings, strategies as st  # noqa: E402


@st.composite
def plan_case(draw):
    sched = draw(st.sampled_from(["butterfly", "butterfly", "ring"]))
    if sched == "ring":
        P = draw(st.integers(1, 40))
        group, k = "cyclic", 2 * (P - 1)
    else:
        group = draw(st.sampled_from(["cyclic", "xor"]))
        P = draw(st.sampled_from(POW2)) if group == "xor" else draw(st.integers(1, 128))
        k = draw(st.sampled_from(ks(P)))
    n = draw(st.integers(0, 3 * P + 7))
    seed = draw(st.integers(0, 2**31 - 1))
    return group, sched, P, k, n, seed


@settings(max_examples=60, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(plan_case())
def test_random_plans_reproduce_oracle(case):
    group, sched, P, k, n, seed = case
    x = np.random.default_rng(seed).integers(-2**31, 2**31, size=(P, n), dtype=np.int64).astype(np.int32)
    plan = ar.Plan(P, n, "int32", "sum", k, group=group, schedule=sched)
    want = oracle.allreduce(x, k, "sum", group=group, schedule=sched)
    got = interpret(plan, x, "sum", "reverse")
    assert np.array_equal(got, want), case
    st_ = plan.stats()
    assert st_.rs_steps + st_.ag_steps == k
    assert st_.bytes_pulled_total == st_.blocks_pulled_per_rank * n * 4


@pytest.mark.parametrize("P,n,k,group,schedule,launches,flat", [
    (128, 128 * 18, 14, "xor", "butterfly", 2, 1),      # Recursive Halving, flat columns: reduce, then broadcast
    (64, 64 * 18, 12, "xor", "butterfly", 2, 1),
    (32, 32 * 18, 10, "xor", "butterfly", 1, 1),        # below 64 ranks: one launch
    (128, 128 * 18, 10, "xor", "butterfly", 1, 1),      # hybrid: the ranks receive different results
    (127, 127 * 18, 14, "cyclic", "butterfly", 2, 1),   # rank slots, split
    (127, 127 * 18, 252, "cyclic", "ring", 2, 1),
    (127, 127 * 18, 11, "cyclic", "butterfly", 1, 1),   # shifted: the ranks receive different results
    (37, 37 * 18, 12, "cyclic", "butterfly", 2, 1),     # rank slots split from 33 ranks up
    (32, 32 * 18, 10, "cyclic", "butterfly", 1, 1),
    (37, 37 * 100, 12, "cyclic", "butterfly", 2, 1),    # long blocks below 256 MiB: rank slots too
    (127, 127 * 100, 14, "cyclic", "butterfly", 2, 1),
    (127, 127 * 100, 252, "cyclic", "ring", 2, 1),
    (4, 4 * 100, 4, "cyclic", "butterfly", 1, 0),       # unsplit, below 33 ranks: block tiles
    (24, 1 << 24, 10, "cyclic", "butterfly", 2, 0),     # block tiles split from 24 ranks at 32 MiB
    (24, 1 << 24, 46, "cyclic", "ring", 2, 0),
    (24, 1 << 23, 10, "cyclic", "butterfly", 2, 0),
    (24, (1 << 23) - 1024, 10, "cyclic", "butterfly", 1, 0),
    (23, 1 << 24, 10, "cyclic", "butterfly", 1, 0),
    (32, 1 << 24, 10, "cyclic", "butterfly", 2, 0),
    (33, 1 << 24, 12, "cyclic", "butterfly", 2, 1),
    (127, 1 << 26, 14, "cyclic", "butterfly", 2, 0),    # 256 MiB per rank: block tiles, split
    (37, 1 << 26, 12, "cyclic", "butterfly", 2, 0),     # block tiles, 256 MiB
    (24, 1 << 26, 10, "cyclic", "butterfly", 2, 0),
    (37, 1 << 22, 8, "cyclic", "butterfly", 1, 1),      # shifted sums at P = 24-48 up to 32 MiB: rank slots
    (37, 1 << 24, 8, "cyclic", "butterfly", 1, 0),
    (127, 1 << 26, 10, "cyclic", "butterfly", 1, 1),    # shifted sums at odd P >= 97: rank slots
    (126, 1 << 26, 10, "cyclic", "butterfly", 1, 0),
])
def test_default_split_of_one_result_plans(P, n, k, group, schedule, launches, flat):
    st = ar.Plan(P, n, "float32", "sum", k, group=group, schedule=schedule).stats()
    assert st.fused_launches == launches
    assert st.fused_flat == flat
    assert st.hbm_bytes_fused == (2 * P + (launches == 2)) * n * 4


@pytest.mark.parametrize("P,n,k,flat", [
    (37, 1 << 22, 8, 1),       # shifted max at P = 24-48 up to 32 MiB: rank slots, as for sums
    (37, 1 << 22, 11, 1),
    (24, 1 << 21, 7, 1),
    (37, 1 << 24, 8, 0),       # 64 MiB: block tiles
    (49, 1 << 22, 8, 0),       # outside the P range of the shifted max instantiations
    (127, 1 << 26, 10, 0),     # shifted sums there take rank slots, max keeps block tiles
    (37, 1 << 22, 12, 1),      # bandwidth-optimal: rank slots from 33 ranks below 256 MiB
])
def test_default_layout_of_max_plans(P, n, k, flat):
    for dtype in ("float32", "int32"):
        st = ar.Plan(P, n, dtype, "max", k).stats()
        assert st.fused_flat == flat, (P, n, k, dtype)


@pytest.mark.parametrize("P,n,k,op,flat", [
    (32, 1 << 24, 10, "sum", 1),    # Recursive Halving on long blocks: flat columns
    (32, 1 << 24, 7, "sum", 1),     # hybrid
    (32, 1 << 24, 7, "max", 1),
    (128, 1 << 22, 14, "max", 1),
    (32, 1 << 24, 5, "sum", 0),     # Recursive Doubling keeps block tiles
    (32, 1 << 24, 5, "max", 0),
    (8, 1 << 24, 6, "sum", 1),
])
def test_xor_plans_on_long_blocks_take_flat_columns(P, n, k, op, flat, monkeypatch):
    st = ar.Plan(P, n, "float32", op, k, group="xor").stats()
    assert st.fused_flat == flat
    monkeypatch.setenv("AR_FUSED_ROTATE", "0")
    assert ar.Plan(P, n, "float32", op, k, group="xor").stats().fused_flat == 0


@pytest.mark.parametrize("P,k,group,schedule,flat", [
    (24, 10, "cyclic", "butterfly", 1), (127, 14, "cyclic", "butterfly", 1), (24, 46, "cyclic", "ring", 1),
    (24, 7, "cyclic", "butterfly", 1), (48, 8, "cyclic", "butterfly", 1),  # shifted max at P = 24-48: rank slots
    (23, 7, "cyclic", "butterfly", 0), (49, 8, "cyclic", "butterfly", 0), (127, 10, "cyclic", "butterfly", 0),
    (32, 10, "xor", "butterfly", 1), (32, 7, "xor", "butterfly", 1),
    (12, 4, "cyclic", "butterfly", 0),
])
def test_max_with_short_blocks_on_flat_columns(P, k, group, schedule, flat):
    for dtype in ("float32", "int32"):
        st = ar.Plan(P, 18 * P, dtype, "max", k, group=group, schedule=schedule).stats()
        assert st.fused_flat == flat, (P, k, group, schedule, dtype)
