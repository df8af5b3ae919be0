"""The plan dump (ar_plan_dump, AR_LOG=1) and the timed execute's host side.

The dump must say what the plan is -- P, n, k, L, r, w and the step counts
of the schedule -- and its launch lines must list exactly the ranges of the
launch tables (ar_plan_launch).  ar_execute_timed must check its arguments
before any device work and report a missing GPU like ar_execute.
"""
import ctypes
import os
import re
import subprocess
import sys

import pytest

from paper_2004_09362_amd import ar

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
B = r"([UXY-])"
RANGE = re.compile(r"\[p (\d+)\.\.(\d+) (copy|reduce2|reduce) from x(\^\d+|[+-]\d+): " + B + " = " + B +
                   r"(?: \(\+\) " + B + r")?(?:, " + B + " = " + B + r" \(\+\) " + B + r")?\]")
BUF = {"U": 0, "X": 1, "Y": 2, "-": -1}
KIND = {"copy": 0, "reduce": 1, "reduce2": 2}


def ceil_log2(P):
    return max(0, (P - 1).bit_length())


def parse_launch_line(line):
    out = []
    for m in RANGE.finditer(line):
        p0, p1, kind, dst = int(m[1]), int(m[2]), KIND[m[3]], BUF[m[5]]
        delta = int(m[4][1:]) if m[4][0] == "^" else int(m[4])
        if kind == 0:
            own, src = -1, BUF[m[6]]
        else:
            own, src = BUF[m[6]], BUF[m[7]]
        dst2 = own2 = -1
        if kind == 2:
            dst2, own2 = BUF[m[8]], BUF[m[9]]
            assert BUF[m[10]] == src
        out.append(dict(p0=p0, count=p1 - p0 + 1, kind=kind, delta=delta, dst=dst, own=own, dst2=dst2, own2=own2,
                        src=src))
    return out


@pytest.mark.parametrize("P,k,group,schedule", [(7, 5, "cyclic", "butterfly"), (7, 6, "cyclic", "butterfly"),
                                                (12, 4, "cyclic", "butterfly"), (37, 8, "cyclic", "butterfly"),
                                                (2, 1, "cyclic", "butterfly"), (8, 4, "xor", "butterfly"),
                                                (16, 6, "xor", "butterfly"), (5, 8, "cyclic", "ring"),
                                                (1, 0, "cyclic", "butterfly"), (127, 10, "cyclic", "butterfly")])
def test_dump_matches_plan_and_tables(P, k, group, schedule):
    plan = ar.Plan(P, 1000, "float32", "sum", k, group=group, schedule=schedule)
    st = plan.stats()
    text = plan.dump()
    lines = text.rstrip("\n").split("\n")
    launches = plan.launches()
    assert len(lines) == 3 + len(launches)
    L = ceil_log2(P)
    r = 0 if schedule == "ring" else 2 * L - k
    head = "ar_plan P=%d n=1000 dtype=float32 op=sum group=%s schedule=%s k=%d L=%d r=%d w=%d" % (
        P, group, schedule, k, L, r, st.w)
    assert lines[0] == head
    assert "%d reduction + %d distribution" % (st.rs_steps, st.ag_steps) in lines[1]
    assert "%d blocks pulled" % st.blocks_pulled_per_rank in lines[1]
    for i, (phase, ranges) in enumerate(launches):
        assert lines[3 + i].startswith("  launch %d (%s):" % (i, ("reduce", "distribute", "local copy")[phase]))
        assert parse_launch_line(lines[3 + i]) == ranges, (P, k, i)


def test_dump_truncates_into_small_buffers():
    plan = ar.Plan(7, 1000, "int32", "max", 4)
    full = plan.dump()
    n = ctypes.c_int64()
    for cap in (1, 2, 10, len(full), len(full) + 1, len(full) + 50):
        buf = ctypes.create_string_buffer(b"\x7f" * (cap + 8), cap + 8)
        assert ar.lib.ar_plan_dump(plan.handle, buf, cap, ctypes.byref(n)) == ar.AR_OK
        assert n.value == len(full)
        got = buf.raw[:cap + 8]
        k = min(len(full), cap - 1)
        assert got[:k].decode() == full[:k] and got[k] == 0
        assert got[cap:] == b"\x7f" * 8  # nothing written past cap
    assert ar.lib.ar_plan_dump(plan.handle, None, 0, ctypes.byref(n)) == ar.AR_OK and n.value == len(full)
    assert ar.lib.ar_plan_dump(plan.handle, None, 5, ctypes.byref(n)) == ar.AR_ERR_INVALID_ARG
    assert ar.lib.ar_plan_dump(plan.handle, ctypes.create_string_buffer(4), -1, ctypes.byref(n)) == ar.AR_ERR_INVALID_ARG
    assert ar.lib.ar_plan_dump(None, None, 0, ctypes.byref(n)) == ar.AR_ERR_INVALID_ARG
    assert ar.lib.ar_plan_dump(plan.handle, None, 0, None) == ar.AR_ERR_INVALID_ARG


def test_ar_log_prints_each_plan_to_stderr():
    code = ("import sys; sys.path.insert(0, %r); from paper_2004_09362_amd import ar; "
            "p = ar.Plan(5, 100, 'float32', 'sum', 4); print(p.dump(), end='')" % ROOT)
    env = dict(os.environ, AR_LOG="1")
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stderr
    assert res.stdout and res.stdout in res.stderr
    env.pop("AR_LOG")
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0 and "ar_plan P=5" not in res.stderr


def test_timed_execute_checks_arguments_first():
    plan = ar.Plan(3, 8, "int32", "sum", 2)
    tbl = (ctypes.c_void_p * 3)(0x10000, 0x20000, 0x30000)
    ms = (ctypes.c_float * 4)()
    n = ctypes.c_int32(-1)
    L = ar.lib
    assert L.ar_execute_timed(plan.handle, tbl, 1, 8, None, ms, 4, None) == ar.AR_ERR_INVALID_ARG
    assert L.ar_execute_timed(plan.handle, tbl, 1, 8, None, ms, -1, ctypes.byref(n)) == ar.AR_ERR_INVALID_ARG
    assert L.ar_execute_timed(plan.handle, tbl, 1, 8, None, None, 4, ctypes.byref(n)) == ar.AR_ERR_INVALID_ARG
    assert L.ar_execute_timed(None, tbl, 1, 8, None, ms, 4, ctypes.byref(n)) == ar.AR_ERR_INVALID_ARG
    bad = (ctypes.c_void_p * 3)(0x10000, 0x10010, 0x30000)   # overlapping ranks
    assert L.ar_execute_timed(plan.handle, bad, 1, 8, None, ms, 4, ctypes.byref(n)) == ar.AR_ERR_ALIAS
    assert n.value == 0


def test_timed_execute_without_gpu_reports_no_device():
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("only meaningful on a machine without a GPU")
    plan = ar.Plan(3, 8, "int32", "sum", 2)
    tbl = (ctypes.c_void_p * 3)(0x10000, 0x20000, 0x30000)
    ms = (ctypes.c_float * 4)()
    n = ctypes.c_int32(-1)
    assert ar.lib.ar_execute_timed(plan.handle, tbl, 1, 8, None, ms, 4, ctypes.byref(n)) == ar.AR_ERR_NO_DEVICE
    assert n.value == 0
    # n = 0: nothing to launch, no device needed
    p0 = ar.Plan(3, 0, "int32", "sum", 2)
    assert ar.lib.ar_execute_timed(p0.handle, tbl, 1, 0, None, ms, 4, ctypes.byref(n)) == ar.AR_OK
    assert n.value == 0
