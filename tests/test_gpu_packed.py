"""Packed column tiles against blocked ones, and merged step launches against
block-by-block ones, on the GPU, through the C ABI.

When blocks are short (many small instances), a column-fused wave takes one
block of several instances instead of one block of one instance, so that
its lanes stay busy while the rank rotation, which depends on the block
only, stays uniform.  Every kind of column launch -- bandwidth-optimal
(single and split into reduce plus broadcast), shifted, the XOR group's
halving and hybrid schedules, the Ring -- must give the oracle's bits with
packed tiles (AR_FUSED_PACKED=1), with blocked tiles (=0) and by default,
on batches with gaps between instances, ragged last tile groups and blocks
of zero, one or a few elements, and must leave the gaps untouched.

Sums also run such batches on flat columns (AR_FUSED_ROTATE), every rank's
row loaded whole: the cyclic butterfly plans with r < L and the Ring in a
rank-slot kernel that rotates each lane's column by its block, the XOR
group's plans with the block left out (it only orders the operands of a
halving pair, which a sum does not see).  It is checked forced on and off, with
either tiling, on blocks of every length up to 70 elements (longer blocks
leave most stages of the rotation network unused by a whole wave), and on
seeded random plans with long blocks (65 to about 600 elements), where the
defaults take the rank-slot kernel for some shapes and block tiles for the
rest.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar
from test_gpu_parity import DEV, bits, note

pytestmark = pytest.mark.gpu

# P, n, batch, instance stride, k, group, schedule, op ("isum", "imax": int32 sum, max)
CASES = [
    (5, 23, 37, 29, 6, "cyclic", "butterfly", "sum"),        # bandwidth-optimal, blocks of 4-5, 12 per wave
    (24, 100, 50, 104, 10, "cyclic", "butterfly", "sum"),    # bandwidth-optimal, blocks of 4-5
    (24, 100, 50, 104, 7, "cyclic", "butterfly", "sum"),     # shifted, r = 3
    (37, 300, 20, 301, 8, "cyclic", "butterfly", "sum"),     # shifted prime, blocks of 8-9
    (37, 300, 20, 301, 8, "cyclic", "butterfly", "max"),
    (37, 20, 10, 20, 12, "cyclic", "butterfly", "sum"),      # n < P: blocks of 0 or 1 element
    (64, 700, 11, 701, 12, "cyclic", "butterfly", "sum"),    # split: reduce plus broadcast
    (127, 1000, 9, 1003, 10, "cyclic", "butterfly", "sum"),  # shifted at P = 127, blocks of 7-8
    (127, 1000, 9, 1003, 14, "cyclic", "butterfly", "sum"),  # split at P = 127
    (32, 200, 13, 200, 10, "xor", "butterfly", "sum"),       # Recursive Halving
    (32, 200, 13, 200, 7, "xor", "butterfly", "sum"),        # XOR hybrid, r = 3
    (128, 1000, 5, 1000, 14, "xor", "butterfly", "max"),     # Recursive Halving, split
    (24, 100, 17, 100, 46, "cyclic", "ring", "sum"),         # Ring
    (127, 500, 7, 500, 252, "cyclic", "ring", "sum"),        # Ring, split
    (24, 1200, 6, 1200, 10, "cyclic", "butterfly", "sum"),   # blocks of 50: one instance per packed wave
    (24, 1700, 4, 1700, 10, "cyclic", "butterfly", "sum"),   # blocks of 70: blocked tiles even when forced
    (24, 1700, 4, 1703, 7, "cyclic", "butterfly", "max"),    # shifted, blocks of 70
    (2, 9, 50, 11, 2, "cyclic", "butterfly", "sum"),         # P = 2: one step each way
    (3, 50, 40, 53, 3, "cyclic", "butterfly", "sum"),        # P = 3, r = 1
    (127, 1000, 9, 1003, 8, "cyclic", "butterfly", "sum"),   # shifted at P = 127, r = 6 = L - 1
    (127, 1000, 9, 1003, 13, "cyclic", "butterfly", "sum"),  # shifted at P = 127, r = 1
    (100, 6400, 3, 6400, 12, "cyclic", "butterfly", "sum"),  # blocks of exactly 64
    (37, 300, 20, 301, 9, "cyclic", "butterfly", "isum"),    # int32, shifted
    (127, 1000, 9, 1003, 14, "cyclic", "butterfly", "isum"), # int32, bandwidth-optimal
    (16, 100, 9, 103, 5, "xor", "butterfly", "isum"),        # int32, XOR hybrid
    (64, 300, 6, 300, 12, "xor", "butterfly", "sum"),        # Recursive Halving at P = 64
    (24, 100, 17, 100, 46, "cyclic", "ring", "isum"),        # int32, Ring
    (24, 100, 50, 104, 10, "cyclic", "butterfly", "max"),    # max, bandwidth-optimal: rank slots
    (127, 1000, 9, 1003, 14, "cyclic", "butterfly", "max"),  # max at P = 127, split
    (24, 100, 17, 100, 46, "cyclic", "ring", "max"),         # max, Ring
    (48, 1000, 5, 1001, 94, "cyclic", "ring", "max"),        # max, Ring, split
    (32, 200, 13, 200, 10, "xor", "butterfly", "max"),       # XOR max, flat: each lane's block orders the pairs
    (32, 200, 13, 200, 7, "xor", "butterfly", "max"),        # XOR max, hybrid r = 3
    (128, 2000, 5, 2003, 14, "xor", "butterfly", "max"),     # XOR max, flat, split
    (37, 300, 20, 301, 9, "cyclic", "butterfly", "max"),     # shifted max at P = 24-48: rank slots
    (48, 4000, 3, 4003, 8, "cyclic", "butterfly", "imax"),   # int32 shifted max, blocks of 83-84
    (24, 1700, 4, 1703, 9, "cyclic", "butterfly", "imax"),   # r = 4 = L - 1
]

SETTINGS = [  # AR_FUSED_ROTATE, AR_FUSED_PACKED (None: unset, the default)
    ("0", "0"), ("0", "1"), ("1", None), (None, None),
]


@pytest.mark.parametrize("P,n,B,stride,k,group,schedule,op", CASES)
def test_packed_and_blocked_tiles_agree_with_oracle(P, n, B, stride, k, group, schedule, op, monkeypatch):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    rng = np.random.default_rng(P * 1000 + n + k)
    dtype = "int32" if op in ("isum", "imax") else "float32"
    if dtype == "int32":
        op = op[1:]
        x = rng.integers(-2**31, 2**31, size=(P, B, stride), dtype=np.int64).astype(np.int32)
    else:
        x = rng.normal(size=(P, B, stride)).astype(np.float32)
    want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), k, op, group=group, schedule=schedule)
    if dtype == "int32" and op == "sum":  # wrapping sum, exact whatever the order
        s64 = x[:, :, :n].astype(np.int64).sum(axis=0)
        assert np.array_equal(want, np.broadcast_to(((s64 + 2**31) % 2**32 - 2**31).astype(np.int32), want.shape))
    if op == "max":
        assert np.array_equal(want, np.broadcast_to(x[:, :, :n].max(axis=0), want.shape))
    for rotate, packed in SETTINGS:
        for var, val in (("AR_FUSED_ROTATE", rotate), ("AR_FUSED_PACKED", packed)):
            if val is None:
                monkeypatch.delenv(var, raising=False)
            else:
                monkeypatch.setenv(var, val)
        mode = "rotate=%s packed=%s" % (rotate, packed)
        note("%s %s/%s P=%d n=%d B=%d k=%d op=%s" % (mode, group, schedule, P, n, B, k, op))
        plan = ar.Plan(P, n, dtype, op, k, path=ar.AR_PATH_FUSED, group=group, schedule=schedule)
        X = torch.from_numpy(x).to(DEV)
        plan.batched([X[i] for i in range(P)], B, stride)
        torch.cuda.synchronize()
        got = X.cpu().numpy()
        plan.close()
        assert np.array_equal(bits(got[:, :, :n]), bits(want)), mode
        assert np.array_equal(bits(got[:, :, n:]), bits(x[:, :, n:])), mode


def _random_cases(count, seed):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        group = ["cyclic", "cyclic", "xor", "ring"][rng.integers(4)]
        if group == "xor":
            P = int(2 ** rng.integers(1, 8))
        else:
            P = int(rng.integers(2, 129))
        L = max(0, (P - 1).bit_length())
        if group == "ring":
            k, schedule, group = 2 * (P - 1), "ring", "cyclic"
        else:
            k, schedule = int(rng.integers(L, 2 * L + 1)), "butterfly"
        n = int(rng.integers(1, 70 * P))           # blocks of 0 to 70 elements
        B = int(rng.integers(1, 9))
        stride = n + int(rng.integers(0, 5))
        op = ["sum", "sum", "isum", "max"][rng.integers(4)]
        out.append((P, n, B, stride, k, group, schedule, op))
    return out


@pytest.mark.parametrize("P,n,B,stride,k,group,schedule,op", _random_cases(40, 20261202))
def test_random_short_block_batches(P, n, B, stride, k, group, schedule, op, monkeypatch):
    """Seeded random groups, schedules, P, k, n (blocks of up to 70
    elements), batch sizes and strides, under the default and with flat
    columns forced on and off: the oracle's bits every time."""
    test_packed_and_blocked_tiles_agree_with_oracle(P, n, B, stride, k, group, schedule, op, monkeypatch)


def _random_long_cases(count, seed):
    """Like _random_cases, with blocks of 65 to about 600 elements."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        group = ["cyclic", "cyclic", "xor", "ring"][rng.integers(4)]
        P = int(2 ** rng.integers(1, 8)) if group == "xor" else int(rng.integers(2, 129))
        L = max(0, (P - 1).bit_length())
        if group == "ring":
            k, schedule, group = 2 * (P - 1), "ring", "cyclic"
        else:
            k, schedule = int(rng.integers(L, 2 * L + 1)), "butterfly"
        n = P * int(rng.integers(65, 600)) + int(rng.integers(0, P))
        B = int(rng.integers(1, 4))
        stride = n + int(rng.integers(0, 5))
        op = ["sum", "isum", "max", "imax"][rng.integers(4)]
        out.append((P, n, B, stride, k, group, schedule, op))
    return out


@pytest.mark.parametrize("P,n,B,stride,k,group,schedule,op", _random_long_cases(24, 20261205))
def test_random_long_block_batches(P, n, B, stride, k, group, schedule, op, monkeypatch):
    """Seeded random plans with long blocks (65 to about 600 elements),
    under the default (rank slots where the size rules pick them, block
    tiles elsewhere) and with flat columns forced on and off: the oracle's
    bits every time, gaps untouched."""
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    rng = np.random.default_rng(P * 13 + n + k)
    dtype = "int32" if op in ("isum", "imax") else "float32"
    if dtype == "int32":
        op = op[1:]
        x = rng.integers(-2**31, 2**31, size=(P, B, stride), dtype=np.int64).astype(np.int32)
    else:
        x = rng.normal(size=(P, B, stride)).astype(np.float32)
    want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), k, op, group=group, schedule=schedule)
    for rotate in (None, "0", "1"):
        if rotate is None:
            monkeypatch.delenv("AR_FUSED_ROTATE", raising=False)
        else:
            monkeypatch.setenv("AR_FUSED_ROTATE", rotate)
        plan = ar.Plan(P, n, dtype, op, k, path=ar.AR_PATH_FUSED, group=group, schedule=schedule)
        st = plan.stats()
        note("long blocks rotate=%s %s/%s P=%d n=%d B=%d k=%d %s %s: flat %d, launches %d"
             % (rotate, group, schedule, P, n, B, k, dtype, op, st.fused_flat, st.fused_launches))
        X = torch.from_numpy(x).to(DEV)
        plan.batched([X[i] for i in range(P)], B, stride)
        torch.cuda.synchronize()
        got = X.cpu().numpy()
        plan.close()
        assert np.array_equal(bits(got[:, :, :n]), bits(want)), rotate
        assert np.array_equal(bits(got[:, :, n:]), bits(x[:, :, n:])), rotate


@pytest.mark.parametrize("P,n,B,stride,k,group,schedule,op", _random_cases(24, 20261204))
def test_random_batches_with_the_split_forced_either_way(P, n, B, stride, k, group, schedule, op, monkeypatch):
    """Seeded random plans with AR_FUSED_SPLIT forced off and on (where every
    rank receives the same result: reduce on rank 0 or the block's rank, then
    broadcast), with either kind of broadcast store: the oracle's bits, gaps
    untouched."""
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    rng = np.random.default_rng(P * 11 + n + k)
    dtype = "int32" if op in ("isum", "imax") else "float32"
    if dtype == "int32":
        op = op[1:]
        x = rng.integers(-2**31, 2**31, size=(P, B, stride), dtype=np.int64).astype(np.int32)
    else:
        x = rng.normal(size=(P, B, stride)).astype(np.float32)
    want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), k, op, group=group, schedule=schedule)
    for split, bnt in (("0", "0"), ("1", "0"), ("1", "1")):
        monkeypatch.setenv("AR_FUSED_SPLIT", split)
        monkeypatch.setenv("AR_BCAST_NT", bnt)
        note("split=%s nt=%s %s/%s P=%d n=%d B=%d k=%d op=%s" % (split, bnt, group, schedule, P, n, B, k, op))
        plan = ar.Plan(P, n, dtype, op, k, path=ar.AR_PATH_FUSED, group=group, schedule=schedule)
        X = torch.from_numpy(x).to(DEV)
        plan.batched([X[i] for i in range(P)], B, stride)
        torch.cuda.synchronize()
        got = X.cpu().numpy()
        plan.close()
        assert np.array_equal(bits(got[:, :, :n]), bits(want)), (split, bnt)
        assert np.array_equal(bits(got[:, :, n:]), bits(x[:, :, n:])), (split, bnt)


@pytest.mark.parametrize("P,n,B,k,group,schedule", [
    (32, 200, 13, 10, "xor", "butterfly"), (32, 200, 13, 7, "xor", "butterfly"), (128, 2000, 5, 14, "xor", "butterfly"),
    (24, 100, 17, 10, "cyclic", "butterfly"), (24, 100, 17, 46, "cyclic", "ring"), (127, 1000, 9, 14, "cyclic", "butterfly"),
    (37, 300, 9, 8, "cyclic", "butterfly"), (48, 4000, 3, 9, "cyclic", "butterfly"),  # shifted max in rank slots
    (32, 32 * 300 + 7, 2, 7, "xor", "butterfly"), (64, 64 * 500, 1, 12, "xor", "butterfly"),  # XOR, long blocks
])
def test_max_of_signed_zeros_follows_the_schedules_operand_order(P, n, B, k, group, schedule, monkeypatch):
    """Inputs of +0.0 and -0.0 only: a max of two zeros returns the kept
    operand, so the result bits show whether every combine took its operands
    in the schedule's order -- on flat columns (each lane's own block) and on
    packed tiles alike."""
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    rng = np.random.default_rng(P + n + k)
    x = np.where(rng.integers(0, 2, size=(P, B, n)) == 1, np.float32(-0.0), np.float32(0.0)).astype(np.float32)
    want = oracle.allreduce_batched(x, k, "max", group=group, schedule=schedule)
    assert np.unique(bits(want)).size == 2  # both zeros occur among the results
    for rotate in ("0", "1"):
        monkeypatch.setenv("AR_FUSED_ROTATE", rotate)
        plan = ar.Plan(P, n, "float32", "max", k, path=ar.AR_PATH_FUSED, group=group, schedule=schedule)
        note("signed zeros rotate=%s %s/%s P=%d k=%d flat=%d" % (rotate, group, schedule, P, k, plan.stats().fused_flat))
        X = torch.from_numpy(x).to(DEV)
        plan.batched([X[i] for i in range(P)], B, n)
        torch.cuda.synchronize()
        got = X.cpu().numpy()
        plan.close()
        assert np.array_equal(bits(got), bits(want)), rotate


# ---------------------------------------------------------------------------
# Step-wise path: merged runs of blocks (AR_STEP_MERGE)
# ---------------------------------------------------------------------------

MERGE_CASES = _random_cases(30, 20261203) + [
    (37, 40000, 2, 40007, 9, "cyclic", "butterfly", "sum"),   # blocks of 1081: block tiles by default
    (24, 5000, 3, 5003, 7, "cyclic", "butterfly", "isum"),    # shifted, blocks of 208
    (64, 9000, 2, 9000, 9, "xor", "butterfly", "sum"),        # XOR hybrid, aligned ranges
    (2, 100, 5, 100, 1, "cyclic", "butterfly", "sum"),        # P = 2, k = 1: the local copy launch
    (13, 13 * 64, 4, 13 * 64 + 1, 8, "cyclic", "butterfly", "max"),
]


@pytest.mark.parametrize("P,n,B,stride,k,group,schedule,op", MERGE_CASES)
def test_stepwise_merged_runs_agree_with_oracle(P, n, B, stride, k, group, schedule, op, monkeypatch):
    """One step launch per communication step, with every range streamed as
    one run of blocks per rank (AR_STEP_MERGE=1), block by block (=0) and by
    default: the oracle's bits every time, gaps between instances untouched."""
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    rng = np.random.default_rng(P * 7 + n + k)
    dtype = "int32" if op in ("isum", "imax") else "float32"
    if dtype == "int32":
        op = op[1:]
        x = rng.integers(-2**31, 2**31, size=(P, B, stride), dtype=np.int64).astype(np.int32)
    else:
        x = rng.normal(size=(P, B, stride)).astype(np.float32)
    want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), k, op, group=group, schedule=schedule)
    for merge in ("0", "1", None):
        if merge is None:
            monkeypatch.delenv("AR_STEP_MERGE", raising=False)
        else:
            monkeypatch.setenv("AR_STEP_MERGE", merge)
        note("step-wise merge=%s %s/%s P=%d n=%d B=%d k=%d op=%s" % (merge, group, schedule, P, n, B, k, op))
        plan = ar.Plan(P, n, dtype, op, k, path=ar.AR_PATH_STEPWISE, group=group, schedule=schedule)
        X = torch.from_numpy(x).to(DEV)
        plan.batched([X[i] for i in range(P)], B, stride)
        torch.cuda.synchronize()
        got = X.cpu().numpy()
        plan.close()
        assert np.array_equal(bits(got[:, :, :n]), bits(want)), merge
        assert np.array_equal(bits(got[:, :, n:]), bits(x[:, :, n:])), merge
