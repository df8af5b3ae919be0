"""GPU parity of the XOR-group and Ring plans against the CPU oracle.

Recursive Halving / hybrid / Recursive Doubling (the butterfly schedules over
the group of Table 1b, power-of-two P) and the Ring of Sec. 6, both on the
step-wise and the fused path, through the C ABI.  The bar is that of the
cyclic plans: int32 and max bit-exact, fp32 sums bit-exact against the
oracle's replay of the same order and within 1e-5 of the fp64 direct sum
relative to sum|V| (the Ring's chain has depth P - 1; (P-1) 2^-24 is
below 1e-5 for every P <= 128).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar, synth
from test_gpu_parity import DEV, assert_fp32_bound, bits, note, sample_cols

pytestmark = pytest.mark.gpu

POW2 = [2, 4, 8, 16, 32, 64, 128]
BOTH = [ar.AR_PATH_STEPWISE, ar.AR_PATH_FUSED]


def ceil_log2(P):
    return max(0, (P - 1).bit_length())


def ks(P):
    L = ceil_log2(P)
    return list(range(L, 2 * L + 1))


@pytest.fixture(autouse=True)
def _gpu_present():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    yield


def run(P, n, dtype, op, k, X, path, group, schedule):
    plan = ar.Plan(P, n, dtype, op, k, path=path, group=group, schedule=schedule)
    plan([X[i] for i in range(P)])
    torch.cuda.synchronize()
    plan.close()


def check(x, k, op, group, schedule, dtype, label):
    P, n = x.shape
    want = oracle.allreduce(x, k, op, group=group, schedule=schedule)
    for path in BOTH:
        note("%s P=%d n=%d k=%d op=%s path=%d" % (label, P, n, k, op, path))
        X = torch.from_numpy(x).to(DEV)
        run(P, n, dtype, op, k, X, path, group, schedule)
        got = X.cpu().numpy()
        assert np.array_equal(bits(got), bits(want)), (label, P, k, op, path)
        if op == "sum" and x.dtype == np.float32:
            assert_fp32_bound(got, x)
        if op != "sum" or x.dtype == np.int32:
            assert np.array_equal(got, np.broadcast_to(oracle.direct(x, op).astype(x.dtype), got.shape))


# ---------------------------------------------------------------------------
# XOR group: Recursive Halving, hybrid, Recursive Doubling
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P", POW2)
def test_xor_fp32_every_k(P):
    rng = np.random.default_rng(300 + P)
    for n in (3 * P + 5, P - 1, 4 * P):
        x = (rng.normal(size=(P, n)) * np.exp2(rng.integers(-6, 6, size=(P, n)))).astype(np.float32)
        for k in ks(P):
            check(x, k, "sum", "xor", "butterfly", "float32", "xor fp32")


@pytest.mark.parametrize("P", POW2)
def test_xor_int32_tags_and_max(P):
    rng = np.random.default_rng(400 + P)
    n = 2 * P + 3
    xi = rng.integers(-2**31, 2**31, size=(P, n), dtype=np.int64).astype(np.int32)
    xf = rng.normal(size=(P, n)).astype(np.float32)
    xf[0, :2] = -0.0
    for k in ks(P):
        check(xi, k, "sum", "xor", "butterfly", "int32", "xor int32")
        check(xi, k, "max", "xor", "butterfly", "int32", "xor imax")
        check(xf, k, "max", "xor", "butterfly", "float32", "xor fmax")
    if P <= 16:
        tags = np.stack([np.full(5 * P + 1, 1 << y, np.int32) for y in range(P)])
        for k in ks(P):
            check(tags, k, "sum", "xor", "butterfly", "int32", "xor tags")


@pytest.mark.parametrize("P,n", [(2, 100003), (8, 100003), (16, 65543), (64, 131079), (128, 262147)])
def test_xor_several_tiles_per_block(P, n):
    rng = np.random.default_rng(n % 1000 + P)
    x = rng.normal(size=(P, n)).astype(np.float32)
    for k in sorted({ks(P)[0], ks(P)[len(ks(P)) // 2], ks(P)[-1]}):
        check(x, k, "sum", "xor", "butterfly", "float32", "xor tiles")


# ---------------------------------------------------------------------------
# Ring
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P", range(2, 129))
def test_ring_fp32_every_P(P):
    rng = np.random.default_rng(500 + P)
    n = 3 * P + 5
    x = (rng.normal(size=(P, n)) * np.exp2(rng.integers(-6, 6, size=(P, n)))).astype(np.float32)
    check(x, 2 * (P - 1), "sum", "cyclic", "ring", "float32", "ring fp32")


@pytest.mark.parametrize("P", [2, 3, 5, 7, 12, 37, 100, 128])
def test_ring_int32_and_max(P):
    rng = np.random.default_rng(600 + P)
    n = 2 * P + 7
    xi = rng.integers(-2**31, 2**31, size=(P, n), dtype=np.int64).astype(np.int32)
    xf = rng.normal(size=(P, n)).astype(np.float32)
    xf[1, :2] = -0.0
    k = 2 * (P - 1)
    check(xi, k, "sum", "cyclic", "ring", "int32", "ring int32")
    check(xi, k, "max", "cyclic", "ring", "int32", "ring imax")
    check(xf, k, "max", "cyclic", "ring", "float32", "ring fmax")
    if P <= 16:
        tags = np.stack([np.full(P + 2, 1 << y, np.int32) for y in range(P)])
        check(tags, k, "sum", "cyclic", "ring", "int32", "ring tags")


@pytest.mark.parametrize("P,n", [(3, 100003), (7, 65543), (17, 70001), (37, 74000)])
def test_ring_several_tiles_per_block(P, n):
    rng = np.random.default_rng(n % 997 + P)
    x = rng.normal(size=(P, n)).astype(np.float32)
    check(x, 2 * (P - 1), "sum", "cyclic", "ring", "float32", "ring tiles")


# ---------------------------------------------------------------------------
# Layout cases shared with the cyclic plans
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("group,schedule,P,k", [("xor", "butterfly", 8, 3), ("xor", "butterfly", 16, 6),
                                                ("xor", "butterfly", 32, 10), ("cyclic", "ring", 5, 8),
                                                ("cyclic", "ring", 12, 22)])
def test_batched_with_gaps(group, schedule, P, k):
    rng = np.random.default_rng(P * 7 + k)
    n, B, stride = 53, 9, 61
    x = rng.normal(size=(P, B, stride)).astype(np.float32)
    want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), k, "sum", group=group, schedule=schedule)
    for path in BOTH:
        note("batched %s/%s P=%d k=%d path=%d" % (group, schedule, P, k, path))
        X = torch.from_numpy(x).to(DEV)
        plan = ar.Plan(P, n, "float32", "sum", k, path=path, group=group, schedule=schedule)
        plan.batched([X[i] for i in range(P)], B, stride)
        torch.cuda.synchronize()
        got = X.cpu().numpy()
        assert np.array_equal(bits(got[:, :, :n]), bits(want)), path
        assert np.array_equal(bits(got[:, :, n:]), bits(x[:, :, n:])), path


@pytest.mark.parametrize("shift", [1, 3])
def test_unaligned_separate_buffers(shift):
    """Rank buffers at 4-byte (not 16-byte) offsets, in separate allocations
    handed over in shuffled memory order."""
    for group, schedule, P, k in (("xor", "butterfly", 8, 4), ("cyclic", "ring", 6, 10)):
        n = 1000 + shift
        rng = np.random.default_rng(shift * 13 + P)
        x = rng.normal(size=(P, n)).astype(np.float32)
        want = oracle.allreduce(x, k, "sum", group=group, schedule=schedule)
        for path in BOTH:
            note("unaligned %s/%s P=%d shift=%d path=%d" % (group, schedule, P, shift, path))
            store = [torch.empty(n + 8, device=DEV) for _ in range(P)][::-1]
            views = [store[i][shift:shift + n] for i in range(P)]
            for i in range(P):
                views[i].copy_(torch.from_numpy(x[i]))
            plan = ar.Plan(P, n, "float32", "sum", k, path=path, group=group, schedule=schedule)
            plan(views)
            torch.cuda.synchronize()
            got = np.stack([v.cpu().numpy() for v in views])
            assert np.array_equal(bits(got), bits(want)), (group, path)


# ---------------------------------------------------------------------------
# Full-size shapes, sampled columns
# ---------------------------------------------------------------------------

def full_size(label, P, n, k, group, schedule, seed, dist):
    note("%s P=%d n=%d k=%d: fill" % (label, P, n, k))
    X = synth.device_ranks(seed, P, n, np.float32, dist, DEV)
    X0 = X.clone()
    cols = sample_cols(n, P, per_block=32, seed=k)
    ct = torch.from_numpy(cols).to(DEV)
    xs = X[:, ct].cpu().numpy()
    want = oracle.allreduce(xs, k, "sum", n=n, cols=cols, group=group, schedule=schedule)
    outs = []
    for path in BOTH:
        X.copy_(X0)
        note("%s P=%d n=%d k=%d path=%d: execute" % (label, P, n, k, path))
        plan = ar.Plan(P, n, "float32", "sum", k, path=path, group=group, schedule=schedule)
        plan([X[i] for i in range(P)])
        torch.cuda.synchronize()
        got = X[:, ct].cpu().numpy()
        assert np.array_equal(bits(got), bits(want)), path
        assert_fp32_bound(got, xs)
        outs.append(X.clone())
        plan.close()
    assert torch.equal(outs[0].view(torch.int32), outs[1].view(torch.int32))
    del X, X0, outs
    torch.cuda.empty_cache()


@pytest.mark.parametrize("k", [5, 8, 10])
def test_xor_gradsync_shape(k):
    """The gradient-sync shape at a power of two: P = 32, n = 16,777,216 fp32."""
    w = synth.WORKLOADS["gradsync"]
    full_size("xor gradsync", 32, w["n"], k, "xor", "butterfly", w["seed"], w["dist"])


def test_ring_gradsync_shape():
    """The gradient-sync shape itself: P = 24, n = 16,777,216 fp32, k = 46."""
    w = synth.WORKLOADS["gradsync"]
    full_size("ring gradsync", 24, w["n"], 46, "cyclic", "ring", w["seed"], w["dist"])


# ---------------------------------------------------------------------------
# Split fused launch (reduce, then broadcast) against the single launch
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P,k,group,schedule", [(5, 6, "cyclic", "butterfly"), (24, 10, "cyclic", "butterfly"),
                                                (64, 12, "cyclic", "butterfly"), (127, 14, "cyclic", "butterfly"),
                                                (8, 6, "xor", "butterfly"), (64, 12, "xor", "butterfly"),
                                                (7, 12, "cyclic", "ring"), (64, 126, "cyclic", "ring")])
def test_split_and_single_fused_launch_agree(P, k, group, schedule, monkeypatch):
    """AR_FUSED_SPLIT forces either form, and AR_BCAST_NT either kind of
    broadcast store; all must give the oracle's bits, on a ragged batch with
    gaps between instances, with block tiles and on flat columns
    (AR_FUSED_ROTATE=1: rank 0 holds every result before the broadcast)."""
    rng = np.random.default_rng(P * 3 + k)
    n, B, stride = 5 * P + 3, 3, 5 * P + 11
    x = rng.normal(size=(P, B, stride)).astype(np.float32)
    want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), k, "sum", group=group, schedule=schedule)
    for (rotate, split, bnt) in [(r, s, b) for r in ("0", "1") for s, b in (("0", "0"), ("1", "0"), ("1", "1"))]:
        monkeypatch.setenv("AR_FUSED_ROTATE", rotate)
        monkeypatch.setenv("AR_FUSED_SPLIT", split)
        monkeypatch.setenv("AR_BCAST_NT", bnt)
        plan = ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_FUSED, group=group, schedule=schedule)
        assert plan.stats().fused_launches == (2 if split == "1" else 1)
        assert plan.stats().fused_flat == int(rotate == "1")
        note("flat=%s split=%s broadcast nt=%s %s/%s P=%d k=%d" % (rotate, split, bnt, group, schedule, P, k))
        X = torch.from_numpy(x).to(DEV)
        plan.batched([X[i] for i in range(P)], B, stride)
        torch.cuda.synchronize()
        got = X.cpu().numpy()
        assert np.array_equal(bits(got[:, :, :n]), bits(want)), (rotate, split, bnt)
        assert np.array_equal(bits(got[:, :, n:]), bits(x[:, :, n:])), (rotate, split, bnt)
        plan.close()


@pytest.mark.parametrize("P,k,group,schedule,B", [(12, 4, "cyclic", "butterfly", 40), (24, 10, "cyclic", "butterfly", 1),
                                                  (37, 8, "cyclic", "butterfly", 1), (64, 12, "cyclic", "butterfly", 1),
                                                  (32, 7, "xor", "butterfly", 1), (24, 46, "cyclic", "ring", 1)])
def test_occupancy_cap_does_not_change_bits(P, k, group, schedule, B, monkeypatch):
    """AR_FUSED_CAP = 0 (no cap), 1 and 5 resident workgroups per CU: the
    launch shape changes, the results must not."""
    rng = np.random.default_rng(P + 17 * k)
    n = 4 * P + 9 if B > 1 else 3000 + P
    x = rng.normal(size=(P, B, n)).astype(np.float32)
    want = oracle.allreduce_batched(x, k, "sum", group=group, schedule=schedule)
    for cap in ("0", "1", "5"):
        monkeypatch.setenv("AR_FUSED_CAP", cap)
        note("cap=%s %s/%s P=%d k=%d" % (cap, group, schedule, P, k))
        X = torch.from_numpy(x).to(DEV)
        plan = ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_FUSED, group=group, schedule=schedule)
        plan.batched([X[i] for i in range(P)], B, n)
        torch.cuda.synchronize()
        assert np.array_equal(bits(X.cpu().numpy()), bits(want)), cap
        plan.close()


@pytest.mark.parametrize("group,schedule,P", [("xor", "butterfly", 2), ("xor", "butterfly", 8), ("xor", "butterfly", 64),
                                              ("cyclic", "ring", 2), ("cyclic", "ring", 5), ("cyclic", "ring", 64)])
def test_degenerate_sizes_other_schedules(group, schedule, P):
    """n = 0 (nothing touched), n = 1 and n < P (empty blocks), n = P, on
    every k of the schedule and both paths."""
    kk = [2 * (P - 1)] if schedule == "ring" else ks(P)
    for n in (0, 1, P - 1, P):
        x = np.random.default_rng(n + P).integers(-1000, 1000, size=(P, n)).astype(np.int32)
        for k in kk:
            want = oracle.allreduce(x, k, "sum", group=group, schedule=schedule)
            for path in BOTH:
                note("degenerate %s/%s P=%d n=%d k=%d path=%d" % (group, schedule, P, n, k, path))
                X = torch.from_numpy(x).to(DEV)
                run(P, n, "int32", "sum", k, X, path, group, schedule)
                assert np.array_equal(X.cpu().numpy(), want), (n, k, path)


def test_single_rank_other_schedules():
    """P = 1: both schedules are the identity (k = 0)."""
    x = np.arange(17, dtype=np.float32)[None, :]
    for group, schedule in (("xor", "butterfly"), ("cyclic", "ring")):
        X = torch.from_numpy(x).to(DEV)
        plan = ar.Plan(1, 17, "float32", "sum", 0, group=group, schedule=schedule)
        assert plan.stats().launches == 0 and plan.stats().fused_ok == 0
        plan([X[0]])
        torch.cuda.synchronize()
        assert np.array_equal(X.cpu().numpy(), x)


@pytest.mark.parametrize("layout", ["0", "default"])
@pytest.mark.parametrize("P,k,schedule", [(48, 12, "butterfly"), (40, 78, "ring"), (33, 12, "butterfly")])
def test_split_from_32_ranks_at_64_mib(P, k, schedule, layout, monkeypatch):
    """One-result plans from P = 32 with 64 MiB rank buffers run as a
    reducing launch plus the destination-major broadcast, on block tiles
    (AR_FUSED_ROTATE=0, split from 32 ranks at this size) and on the
    default rank slots (split from 33): the full-size vector against the
    oracle on sampled columns, and the whole vector against the step-wise
    path."""
    if layout == "0":
        monkeypatch.setenv("AR_FUSED_ROTATE", "0")
    w = synth.WORKLOADS["gradsync"]
    st = ar.Plan(P, w["n"], "float32", "sum", k, path=ar.AR_PATH_FUSED, schedule=schedule).stats()
    assert st.fused_launches == 2 and st.fused_bcast_stream == 1 and st.fused_flat == int(layout == "default")
    full_size("split P=%d %s" % (P, schedule), P, w["n"], k, "cyclic", schedule, w["seed"], w["dist"])
