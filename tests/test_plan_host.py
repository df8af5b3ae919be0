"""Host-side checks of libar.so: exports, argument errors, and the schedule
tables (no GPU needed).

The tables of every launch are executed here by a small numpy interpreter
(test code, not the library) and compared bit for bit with the independent
CPU oracle; running each launch's work items forward, backward and from a
pre-launch snapshot must give the same bits, which is what lets the GPU run
them in any order.
"""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
from paper_2004_09362_amd import ar

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def ceil_log2(P):
    return max(0, (P - 1).bit_length())


def ks(P):
    L = ceil_log2(P)
    return list(range(L, 2 * L + 1))


def header_functions():
    text = open(os.path.join(ROOT, "include", "ar.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ar_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = header_functions()
    assert set(names) == set(ar.EXPORTS)
    for name in names:
        assert hasattr(ar.lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", ar.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (ar_\w+)", out))
    assert set(names) <= exported


def test_library_is_built_for_gfx950_only(tmp_path):
    llvm = "/opt/rocm/llvm/bin/"
    fb = tmp_path / "fatbin"
    subprocess.run([llvm + "llvm-objcopy", "--dump-section", ".hip_fatbin=%s" % fb, ar.LIB_PATH,
                    str(tmp_path / "copy.so")], check=True)
    # one bundle per translation unit, stored compressed ("CCOB" header) or
    # plain; list each on its own
    data = fb.read_bytes()
    starts = sorted(m.start() for m in re.finditer(rb"CCOB|__CLANG_OFFLOAD_BUNDLE__", data))
    assert starts, "no offload bundle in libar.so"
    targets = set()
    for i, s in enumerate(starts):
        part = tmp_path / ("bundle%d" % i)
        part.write_bytes(data[s:starts[i + 1] if i + 1 < len(starts) else len(data)].rstrip(b"\0"))
        out = subprocess.run([llvm + "clang-offload-bundler", "--list", "--type=o", "--input=%s" % part],
                             capture_output=True, text=True, check=True).stdout
        targets |= set(re.findall(r"amdgcn-amd-amdhsa--(gfx\w+)", out))
    assert targets == {"gfx950"}


def test_status_strings():
    for s in range(8):
        assert ar.ar_status_string(s) not in ("", "unknown status")
    assert ar.ar_status_string(99) == "unknown status"


@pytest.mark.parametrize("args,status", [
    ((0, 10, "float32", "sum", 0), ar.AR_ERR_INVALID_ARG),
    ((129, 10, "float32", "sum", 14), ar.AR_ERR_UNSUPPORTED),     # above the compiled maximum
    ((7, -1, "float32", "sum", 3), ar.AR_ERR_INVALID_ARG),
    ((7, 10, "float32", "sum", 2), ar.AR_ERR_INVALID_ARG),
    ((7, 10, "float32", "sum", 7), ar.AR_ERR_INVALID_ARG),
    ((1, 10, "float32", "sum", 1), ar.AR_ERR_INVALID_ARG),
    ((7, (1 << 46) + 1, "float32", "sum", 4), ar.AR_ERR_INVALID_ARG),   # beyond 2^46 elements per rank
])
def test_plan_create_rejects(args, status):
    with pytest.raises(ar.ArError) as ei:
        ar.ar_plan_create(*args)
    assert ei.value.status == status
    assert ar.ar_last_error() != ""


def test_plan_create_rejects_unknown_dtype_and_op():
    h = ctypes.c_void_p()
    assert ar.lib.ar_plan_create(5, 10, 7, 0, 3, ctypes.byref(h)) == ar.AR_ERR_UNSUPPORTED
    assert ar.lib.ar_plan_create(5, 10, 1, 9, 3, ctypes.byref(h)) == ar.AR_ERR_UNSUPPORTED
    assert ar.lib.ar_plan_create(5, 10, 1, 0, 3, None) == ar.AR_ERR_INVALID_ARG


def test_fused_path_for_every_plan_with_two_or_more_ranks():
    for P in range(1, 129):
        L = ceil_log2(P)
        for k in ks(P):
            assert ar.Plan(P, 64, "float32", "sum", k).stats().fused_ok == int(P >= 2), (P, k)
    ar.Plan(12, 106, "float32", "sum", 4).set_path(ar.AR_PATH_FUSED)
    ar.Plan(12, 106, "float32", "sum", 5).set_path(ar.AR_PATH_FUSED)
    with pytest.raises(ar.ArError) as ei:
        ar.Plan(1, 106, "float32", "sum", 0).set_path(ar.AR_PATH_FUSED)
    assert ei.value.status == ar.AR_ERR_UNSUPPORTED


@pytest.mark.parametrize("P,n,k,group,rotate,want", [
    (127, 1 << 26, 14, "cyclic", None, 1),          # split, 256 MiB rank buffers: block tiles
    (64, 1 << 26, 12, "cyclic", None, 1),
    (128, 1 << 26, 14, "xor", None, 1),
    (127, 1 << 25, 14, "cyclic", None, 1),          # below 256 MiB: rank slots (flat columns)
    (127, 1 << 25, 14, "cyclic", "0", 1),           # block tiles, 128 MiB: one region of chunks per XCD
    (127, 1 << 24, 14, "cyclic", "0", 1),           # 64 MiB
    (127, (1 << 24) - 1024, 14, "cyclic", "0", 1),
    (127, 1 << 19, 14, "cyclic", "0", 1),           # 2 MiB
    (127, (1 << 19) - 1024, 14, "cyclic", "0", 0),  # just below 2 MiB: the tiled broadcast
    (127, 127 * 1024, 14, "cyclic", "0", 0),
    (127, (1 << 19) - 1024, 14, "cyclic", None, 1), # the same on rank slots: flat, any size
    (127, 2304, 14, "cyclic", None, 1),             # short blocks on flat columns (results on rank 0)
    (128, 2304, 14, "xor", None, 1),
    (48, 2304, 12, "cyclic", None, 1),              # flat, any P
    (127, 1 << 26, 10, "cyclic", None, 0),          # shifted: one launch, no broadcast
    (37, 1 << 22, 12, "cyclic", "0", 0),            # block tiles below the split's P
    (37, 1 << 22, 12, "cyclic", None, 1),           # rank slots split from 33 ranks
])
def test_destination_major_broadcast_choice(P, n, k, group, rotate, want, monkeypatch):
    if rotate is not None:
        monkeypatch.setenv("AR_FUSED_ROTATE", rotate)
    st = ar.Plan(P, n, "float32", "sum", k, group=group).stats()
    assert st.fused_bcast_stream == want
    assert st.fused_launches == (2 if want else st.fused_launches)
    # the override: never, or wherever the call allows it (split plans with
    # flat columns or blocks of at least 1024 elements)
    monkeypatch.setenv("AR_BCAST_STREAM", "0")
    assert ar.Plan(P, n, "float32", "sum", k, group=group).stats().fused_bcast_stream == 0
    allowed = st.fused_launches == 2 and (st.fused_flat == 1 or n // P >= 1024)
    for mode in ("1", "2", "3"):  # chunk order by size, interleaved, XCD regions
        monkeypatch.setenv("AR_BCAST_STREAM", mode)
        assert ar.Plan(P, n, "float32", "sum", k, group=group).stats().fused_bcast_stream == int(allowed)
    monkeypatch.setenv("AR_BCAST_STREAM", "4")  # not a mode: the size rules
    assert ar.Plan(P, n, "float32", "sum", k, group=group).stats().fused_bcast_stream == want


def test_execute_argument_errors_before_any_device_work():
    p = ar.Plan(3, 8, "int32", "sum", 2)
    tbl = (ctypes.c_void_p * 3)(0x10000, 0, 0x30000)
    assert ar.lib.ar_execute(p.handle, tbl, None) == ar.AR_ERR_INVALID_ARG
    tbl = (ctypes.c_void_p * 3)(0x10000, 0x20002, 0x30000)
    assert ar.lib.ar_execute(p.handle, tbl, None) == ar.AR_ERR_INVALID_ARG
    tbl = (ctypes.c_void_p * 3)(0x10000, 0x10010, 0x30000)   # 8 int32 = 32 bytes: overlap
    assert ar.lib.ar_execute(p.handle, tbl, None) == ar.AR_ERR_ALIAS
    tbl = (ctypes.c_void_p * 3)(0x10000, 0x20000, 0x30000)
    assert ar.lib.ar_execute_batched(p.handle, tbl, 0, 8, None) == ar.AR_ERR_INVALID_ARG
    assert ar.lib.ar_execute_batched(p.handle, tbl, 2, 7, None) == ar.AR_ERR_INVALID_ARG
    assert ar.lib.ar_execute(None, tbl, None) == ar.AR_ERR_INVALID_ARG
    assert ar.lib.ar_execute(p.handle, None, None) == ar.AR_ERR_INVALID_ARG
    # a rank's extent beyond 2^46 elements, including products that overflow 64 bits
    assert ar.lib.ar_execute_batched(p.handle, tbl, 1 << 40, 1 << 30, None) == ar.AR_ERR_INVALID_ARG
    assert ar.lib.ar_execute_batched(p.handle, tbl, (1 << 63) - 1, 8, None) == ar.AR_ERR_INVALID_ARG
    assert ar.lib.ar_execute_batched(p.handle, tbl, (1 << 38) + 1, 1 << 8, None) == ar.AR_ERR_INVALID_ARG


def test_trivial_plans_do_nothing():
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("host-only check")
    p1 = ar.Plan(1, 10, "float32", "sum", 0)
    assert p1.stats().launches == 0
    tbl = (ctypes.c_void_p * 1)(0x10000)
    assert ar.lib.ar_execute(p1.handle, tbl, None) == ar.AR_OK
    p0 = ar.Plan(5, 0, "float32", "sum", 3)
    tbl = (ctypes.c_void_p * 5)(*[0x10000 * (i + 1) for i in range(5)])
    assert ar.lib.ar_execute(p0.handle, tbl, None) == ar.AR_OK


def test_execute_without_gpu_reports_no_device():
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("only meaningful on a machine without a GPU")
    p = ar.Plan(3, 8, "int32", "sum", 2)
    tbl = (ctypes.c_void_p * 3)(0x10000, 0x20000, 0x30000)
    assert ar.lib.ar_execute(p.handle, tbl, None) == ar.AR_ERR_NO_DEVICE


# ---------------------------------------------------------------------------
# The tables against the oracle
# ---------------------------------------------------------------------------

def part(n, P):
    q, m = divmod(n, P)
    lens = [q + (b < m) for b in range(P)]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(int)
    return offs


def comb(op, a, b):
    if op == "sum":
        if a.dtype == np.int32:
            return (a.astype(np.uint32) + b.astype(np.uint32)).astype(np.int32)
        return (a + b).astype(a.dtype)
    return np.where(b > a, b, a)


def interpret(plan, x, op, order="forward"):
    """Run the plan's launch tables on numpy rank buffers (test oracle of the
    tables' semantics as documented in include/ar.h)."""
    P, n = x.shape
    offs = part(n, P)
    xor = plan.stats().group == ar.AR_GROUP_XOR
    bufs = {0: x.copy(), 1: np.zeros_like(x), 2: np.zeros_like(x)}
    for phase, ranges in plan.launches():
        items = []
        for r in ranges:
            for j in range(r["count"]):
                for rank in range(P):
                    items.append((r, (r["p0"] + j) % P, rank))
        if order == "reverse":
            items = items[::-1]
        src_bufs = {k: v.copy() for k, v in bufs.items()} if order == "snapshot" else bufs
        for r, p, rank in items:
            b = (rank ^ p) if xor else (rank - p) % P
            sl = slice(offs[b], offs[b + 1])
            y = (rank ^ r["delta"]) if xor else (rank + r["delta"]) % P
            s = src_bufs[r["src"]][y, sl].copy()
            if r["kind"] == ar.AR_KIND_COPY:
                bufs[r["dst"]][rank, sl] = s
            else:
                own = src_bufs[r["own"]][rank, sl].copy()
                if r["kind"] == ar.AR_KIND_REDUCE2:
                    own2 = src_bufs[r["own2"]][rank, sl].copy()
                    bufs[r["dst2"]][rank, sl] = comb(op, own2, s)
                bufs[r["dst"]][rank, sl] = comb(op, own, s)
    return bufs[0]


@pytest.mark.parametrize("P", list(range(1, 34)) + [37, 48, 63, 64, 65, 100, 127, 128])
def test_plan_sizes_match_oracle_counts(P):
    """Steps, blocks received per step, combinations and bytes of the plan
    equal the oracle's counts of the same schedule."""
    for k in ks(P):
        t = oracle.Terms(P, k)
        tr = t.trace
        plan = ar.Plan(P, 10 * P + 3, "float32", "sum", k)
        st = plan.stats()
        assert (st.rs_steps, st.ag_steps, st.L, st.r, st.w) == (tr.rs_steps, tr.ag_steps, tr.L, tr.r, tr.w)
        assert st.blocks_pulled_per_rank == sum(tr.pulls[:k])
        assert st.combines_per_rank == sum(tr.combines[:tr.rs_steps])
        assert st.bytes_pulled_total == st.blocks_pulled_per_rank * st.n * 4
        split = st.fused_launches == 2
        assert st.fused_launches == (0 if P == 1 else 2 if split else 1)
        # plans whose ranks all receive the same result split: from P = 33 up on flat columns (blocks of 10-11
        # elements, the rank-slot kernel), from P = 64 up on block tiles
        assert split == (P >= 33 and k == 2 * ceil_log2(P))
        assert st.fused_flat == int(P >= 2 and k > ceil_log2(P))
        # blocks of 100 elements: the rank-slot kernel, split, from P = 33 up; block tiles below
        big = ar.Plan(P, 100 * P + 3, "float32", "sum", k).stats()
        assert (big.fused_launches == 2) == (P >= 33 and k == 2 * ceil_log2(P))
        if k == 2 * ceil_log2(P) and P > 1:
            assert big.fused_flat == int(P >= 33)
        assert st.hbm_bytes_fused == ((2 * P + split) * st.n * 4 if P > 1 else 0)
        # per-launch pulls equal the oracle's per-step pulls
        launches = [l for l in plan.launches() if l[0] != 2]
        assert len(launches) == k
        for s, (phase, ranges) in enumerate(launches):
            pulled = {(r["src"], (r["p0"] + j + r["delta"]) % P) for r in ranges if r["delta"] != 0
                      for j in range(r["count"])}
            assert len(pulled) == tr.pulls[s], (P, k, s)
        if k == 2 * ceil_log2(P):  # bandwidth-optimal: 5 (P-1) blocks of HBM traffic per rank
            assert st.hbm_bytes_stepwise == 5 * (P - 1) * st.n * 4
            assert st.workspace_bytes == 0


@pytest.mark.parametrize("P", list(range(1, 20)) + [24, 31, 32, 33, 37])
def test_plan_tables_reproduce_oracle_bits(P):
    rng = np.random.default_rng(1000 + P)
    for k in ks(P):
        plan = ar.Plan(P, 2 * P + 5, "float32", "sum", k)
        for n in (2 * P + 5, P - 1 if P > 1 else 1):
            plan = ar.Plan(P, n, "float32", "sum", k)
            x = rng.normal(size=(P, n)).astype(np.float32) * np.exp2(rng.integers(-8, 8, size=(P, n)))
            x = x.astype(np.float32)
            want = oracle.allreduce(x, k, "sum")
            for order in ("forward", "reverse", "snapshot"):
                got = interpret(plan, x, "sum", order)
                assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), (P, k, n, order)


@pytest.mark.parametrize("P", [3, 5, 6, 12, 37])
def test_plan_tables_int32_and_max(P):
    rng = np.random.default_rng(P)
    n = 3 * P + 2
    xi = rng.integers(-2**31, 2**31, size=(P, n), dtype=np.int64).astype(np.int32)
    for k in ks(P):
        plan = ar.Plan(P, n, "int32", "sum", k)
        assert np.array_equal(interpret(plan, xi, "sum"), oracle.allreduce(xi, k, "sum"))
        plan = ar.Plan(P, n, "int32", "max", k)
        assert np.array_equal(interpret(plan, xi, "max"), oracle.allreduce(xi, k, "max"))


def test_bandwidth_optimal_runs_in_place():
    for P in (2, 3, 24, 37, 127):
        L = ceil_log2(P)
        plan = ar.Plan(P, 1000, "float32", "sum", 2 * L)
        for phase, ranges in plan.launches():
            for r in ranges:
                assert r["dst"] == 0 and r["src"] == 0 and r["own"] in (0, -1)


def test_launch_count_is_k():
    for P in range(2, 129):
        for k in ks(P):
            st = ar.Plan(P, 64, "float32", "sum", k).stats()
            extra = 1 if (P == 2 and k == 1) else 0   # one local copy back into the caller's buffers
            assert st.launches == k + extra
