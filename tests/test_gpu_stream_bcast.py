"""GPU parity of the split plans' two broadcasts against the CPU oracle.

Plans whose ranks all receive one result (bandwidth-optimal in either group,
the Ring) run fused at P >= 64 as a reducing launch plus a broadcast.  The
broadcast can run destination-major when the instances are contiguous and
every rank buffer is 16-byte aligned, with blocks of at least 1024 elements
(or flat columns, whose results all sit on rank 0); otherwise the tiled
kernel copies each block from its root.  By default the library takes the
destination-major copy on flat columns and on rank buffers of 2 MiB and
more, its chunks interleaved over the XCDs or in one contiguous region per
XCD by shape.  A chunk across a block or instance boundary is copied as
whole 16-byte groups, each element from its own root's load (the kernel for
blocks off the 4 KB chunk grid), or element by element (the kernel for
blocks on it, where only the tail takes that path).  Below 256 MiB per rank the
one-result plans take flat columns by default from P = 8 up; the tests run
each case on block tiles too (AR_FUSED_ROTATE=0), which the defaults keep
for larger buffers.  They set AR_BCAST_STREAM (2: interleaved, 3: regions,
1: the default order) so that the copy runs at sizes the oracle checks whole, and compare both copies bit for
bit with the oracle: sizes that span several 4 KB chunks per block, chunks
across block and instance boundaries, and a ragged tail.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def note(msg):
    print("[gpu] " + msg, flush=True)
    sys.stdout.flush()


def bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint32) if a.dtype == np.float32 else a


def draw(rng, P, count, dtype):
    if dtype == "int32":
        return rng.integers(-(1 << 20), 1 << 20, size=(P, count)).astype(np.int32)
    return rng.normal(size=(P, count)).astype(np.float32)


def aligned_rows(x, pad=0):
    """Device copy of x [P, count] whose rows start on 16-byte boundaries
    (row pitch rounded up to 4 elements, plus `pad` elements), and the row
    views of the original length."""
    P, count = x.shape
    pitch = (count + 3) // 4 * 4 + pad
    big = torch.zeros(P, pitch, dtype=torch.int32 if x.dtype == np.int32 else torch.float32, device=DEV)
    big[:, :count] = torch.from_numpy(x).to(DEV)
    return big, [big[i, :count] for i in range(P)]


# P, n, k, group, schedule, dtype, op: blocks of at least 1024 elements (n >= 1024 P)
CASES = [
    (64, 64 * 1024, 12, "cyclic", "butterfly", "float32", "sum"),
    (64, 64 * 1024 + 333, 12, "cyclic", "butterfly", "int32", "max"),
    (127, 127 * 1024 + 77, 14, "cyclic", "butterfly", "float32", "sum"),
    (127, 127 * 1500 + 126, 14, "cyclic", "butterfly", "float32", "max"),
    (128, 128 * 1024 + 5, 14, "xor", "butterfly", "float32", "sum"),
    (100, 100 * 1100 + 3, 198, "cyclic", "ring", "float32", "sum"),
    (64, 64 * 1024 + 63, 12, "cyclic", "butterfly", "float32", "sum"),  # blocks of 1024-1025: a straddle per block
    (37, 2049 * 1024 + 5, 12, "cyclic", "butterfly", "int32", "sum"),   # 2050 chunks: five evened-out slices
]


ORDERS = ["2", "3"]  # interleaved chunks, XCD regions
LAYOUTS = ["0", "default"]  # block tiles (AR_FUSED_ROTATE=0), the default (flat columns from P = 8)


def set_layout(layout, monkeypatch):
    if layout == "default":
        monkeypatch.delenv("AR_FUSED_ROTATE", raising=False)
    else:
        monkeypatch.setenv("AR_FUSED_ROTATE", layout)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("P,n,k,group,schedule,dtype,op", CASES)
def test_split_broadcast_aligned_rows(P, n, k, group, schedule, dtype, op, order, layout, monkeypatch):
    """16-byte aligned rows: the destination-major broadcast (the split
    forced, for P = 37)."""
    monkeypatch.setenv("AR_BCAST_STREAM", order)
    monkeypatch.setenv("AR_FUSED_SPLIT", "1")
    set_layout(layout, monkeypatch)
    rng = np.random.default_rng(P * 7 + n)
    x = draw(rng, P, n, dtype)
    plan = ar.Plan(P, n, dtype, op, k, group=group, schedule=schedule)
    st = plan.stats()
    assert st.fused_launches == 2 and st.exec_path == ar.AR_PATH_FUSED and st.fused_bcast_stream == 1
    if group == "cyclic":
        assert st.fused_flat == int(layout == "default")
    big, views = aligned_rows(x)
    note("stream broadcast P=%d n=%d k=%d %s/%s %s %s order %s layout %s flat %d"
         % (P, n, k, group, schedule, dtype, op, order, layout, st.fused_flat))
    plan(views)
    torch.cuda.synchronize()
    got = big[:, :n].cpu().numpy()
    want = oracle.allreduce(x, k, op, group=group, schedule=schedule)
    assert np.array_equal(bits(got), bits(want))
    assert not big[:, n:].any().item()  # the row padding is never written
    plan.close()


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("P,n,k", [(127, 127 * 1024 + 77, 14), (64, 64 * 1030 + 1, 12)])
def test_split_broadcast_contiguous_batch(P, n, k, order, layout, monkeypatch):
    """Three contiguous instances (stride n) in one buffer per rank: chunks
    that straddle an instance boundary take the last block of one instance
    and the first of the next."""
    monkeypatch.setenv("AR_BCAST_STREAM", order)
    set_layout(layout, monkeypatch)
    B = 3
    rng = np.random.default_rng(P + k)
    x = draw(rng, P, B * n, "float32")
    big, views = aligned_rows(x)
    plan = ar.Plan(P, n, "float32", "sum", k)
    st = plan.stats()
    assert st.fused_launches == 2 and st.fused_bcast_stream == 1 and st.fused_flat == int(layout == "default")
    note("stream broadcast batch P=%d n=%d B=%d k=%d order %s layout %s" % (P, n, B, k, order, layout))
    plan.batched(views, B, n)
    torch.cuda.synchronize()
    got = big[:, :B * n].cpu().numpy().reshape(P, B, n)
    assert np.array_equal(bits(got), bits(oracle.allreduce_batched(x.reshape(P, B, n), k, "sum")))
    plan.close()


def test_tiled_and_stream_broadcasts_agree(monkeypatch):
    """The same plan and input through both broadcasts: aligned rows
    (destination-major), one rank buffer 4 bytes off a 16-byte boundary and
    instances with gaps between them (both tiled); every result equals the
    oracle's bits, and the gaps are left untouched.  Block tiles
    (AR_FUSED_ROTATE=0), whose boundary chunks straddle two roots."""
    monkeypatch.setenv("AR_BCAST_STREAM", "1")
    monkeypatch.setenv("AR_FUSED_ROTATE", "0")
    P, n, k = 127, 127 * 1024 + 501, 14
    rng = np.random.default_rng(2004)
    x = draw(rng, P, n, "float32")
    want = bits(oracle.allreduce(x, k, "sum"))
    plan = ar.Plan(P, n, "float32", "sum", k)
    # aligned rows
    big, views = aligned_rows(x)
    note("broadcasts agree: aligned P=%d n=%d" % (P, n))
    plan(views)
    torch.cuda.synchronize()
    assert np.array_equal(bits(big[:, :n].cpu().numpy()), want)
    # rank 5 one element past a 16-byte boundary
    big, views = aligned_rows(x, pad=4)
    big[5, 1:n + 1] = torch.from_numpy(x[5]).to(DEV)
    views[5] = big[5, 1:n + 1]
    note("broadcasts agree: one unaligned rank P=%d n=%d" % (P, n))
    plan(views)
    torch.cuda.synchronize()
    got = np.stack([v.cpu().numpy() for v in views])
    assert np.array_equal(bits(got), want)
    # two instances with a gap of 12 elements
    B, stride = 2, n + 12
    x2 = draw(rng, P, B * n, "float32").reshape(P, B, n)
    buf = torch.full((P, (B - 1) * stride + n), -7.0, dtype=torch.float32, device=DEV)
    for j in range(B):
        buf[:, j * stride:j * stride + n] = torch.from_numpy(x2[:, j]).to(DEV)
    note("broadcasts agree: gaps P=%d n=%d B=%d" % (P, n, B))
    plan.batched([buf[i] for i in range(P)], B, stride)
    torch.cuda.synchronize()
    h = buf.cpu().numpy()
    got2 = np.stack([h[:, j * stride:j * stride + n] for j in range(B)], axis=1)
    assert np.array_equal(bits(got2), bits(oracle.allreduce_batched(x2, k, "sum")))
    assert np.all(h[:, n:stride] == -7.0)
    plan.close()
    # the same aligned rows through the tiled copy
    monkeypatch.setenv("AR_BCAST_STREAM", "0")
    plan = ar.Plan(P, n, "float32", "sum", k)
    assert plan.stats().fused_bcast_stream == 0
    big, views = aligned_rows(x)
    note("broadcasts agree: aligned, tiled P=%d n=%d" % (P, n))
    plan(views)
    torch.cuda.synchronize()
    assert np.array_equal(bits(big[:, :n].cpu().numpy()), want)
    plan.close()


@pytest.mark.parametrize("order", ["1", "3"])
def test_flat_split_broadcast_small_instances(order, monkeypatch):
    """Short blocks on flat columns (results on rank 0 before the broadcast):
    40 instances of 2304 elements at P = 127, bandwidth-optimal, contiguous;
    chunks interleaved (the default on flat columns) or in XCD regions."""
    monkeypatch.setenv("AR_BCAST_STREAM", order)
    P, n, B, k = 127, 2304, 40, 14
    rng = np.random.default_rng(77)
    x = draw(rng, P, B * n, "float32")
    big, views = aligned_rows(x)
    plan = ar.Plan(P, n, "float32", "sum", k)
    st = plan.stats()
    assert st.fused_flat == 1 and st.fused_launches == 2 and st.fused_bcast_stream == 1
    note("flat stream broadcast P=%d n=%d B=%d order %s" % (P, n, B, order))
    plan.batched(views, B, n)
    torch.cuda.synchronize()
    got = big[:, :B * n].cpu().numpy().reshape(P, B, n)
    assert np.array_equal(bits(got), bits(oracle.allreduce_batched(x.reshape(P, B, n), k, "sum")))
    plan.close()


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("P,k,group,schedule", [
    (2, 2, "cyclic", "butterfly"), (3, 4, "cyclic", "butterfly"), (5, 6, "cyclic", "butterfly"),
    (8, 6, "xor", "butterfly"), (16, 30, "cyclic", "ring"), (17, 10, "cyclic", "butterfly")])
def test_split_forced_at_small_p(P, k, group, schedule, order, layout, monkeypatch):
    """Few destinations: the split forced (AR_FUSED_SPLIT=1) with the
    destination-major copy, blocks of at least 1024 elements off the chunk
    grid, three contiguous instances and a ragged tail."""
    monkeypatch.setenv("AR_FUSED_SPLIT", "1")
    monkeypatch.setenv("AR_BCAST_STREAM", order)
    set_layout(layout, monkeypatch)
    n, B = P * 1500 + 7, 3
    rng = np.random.default_rng(P * 31 + k)
    x = draw(rng, P, B * n, "float32")
    big, views = aligned_rows(x)
    plan = ar.Plan(P, n, "float32", "sum", k, group=group, schedule=schedule)
    st = plan.stats()
    assert st.fused_launches == 2 and st.fused_bcast_stream == 1
    note("forced split P=%d n=%d B=%d k=%d %s/%s order %s" % (P, n, B, k, group, schedule, order))
    plan.batched(views, B, n)
    torch.cuda.synchronize()
    got = big[:, :B * n].cpu().numpy().reshape(P, B, n)
    want = oracle.allreduce_batched(x.reshape(P, B, n), k, "sum", group=group, schedule=schedule)
    assert np.array_equal(bits(got), bits(want))
    plan.close()
