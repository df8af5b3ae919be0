"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bar (element by element, same seeded inputs on both sides):
  - int32 sum and every max: bit-exact (and equal to the plain definition);
  - fp32 sum: bit-exact against the oracle's replay of the same reduction
    order, and within 1e-5 of the fp64 direct sum relative to sum|V|.
Small sizes are compared in full; the full-size workloads on sampled
columns (first, last and random columns of every block), which the oracle
replays one by one.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar, synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def note(msg):
    print("[gpu] " + msg, flush=True)
    sys.stdout.flush()


def ceil_log2(P):
    return max(0, (P - 1).bit_length())


def ks(P):
    L = ceil_log2(P)
    return list(range(L, 2 * L + 1))


def run_plan(P, n, dtype, op, k, X, path=ar.AR_PATH_AUTO):
    """X: [P, n] device tensor, reduced in place through ar_execute."""
    plan = ar.Plan(P, n, dtype, op, k, path=path)
    plan([X[i] for i in range(P)])
    torch.cuda.synchronize()
    plan.close()


def paths(P, k):
    """Every execution path that can run the plan: step-wise always, and the
    single-launch fused kernel where it applies."""
    st = ar.Plan(P, 8, "float32", "sum", k).stats()
    return [ar.AR_PATH_STEPWISE, ar.AR_PATH_FUSED] if st.fused_ok else [ar.AR_PATH_STEPWISE]


def bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint32) if a.dtype == np.float32 else a


def assert_fp32_bound(out, x):
    s64 = x.astype(np.float64).sum(axis=0)
    mag = np.abs(x.astype(np.float64)).sum(axis=0)
    mag[mag == 0] = 1.0
    err = np.abs(out.astype(np.float64) - s64[None, :]) / mag[None, :]
    assert err.max() <= 1e-5, err.max()


def sample_cols(n, P, per_block=64, seed=0):
    q, m = divmod(n, P)
    lens = [q + (b < m) for b in range(P)]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    rng = np.random.default_rng(seed)
    cols = []
    for b in range(P):
        lo, hi = offs[b], offs[b + 1]
        if hi <= lo:
            continue
        cols.extend(range(lo, min(hi, lo + 8)))
        cols.extend(range(max(lo, hi - 8), hi))
        cols.extend(rng.integers(lo, hi, size=per_block).tolist())
    return np.unique(np.array(cols, dtype=np.int64))


@pytest.fixture(autouse=True)
def _gpu_present():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    yield


# ---------------------------------------------------------------------------
# Workload: P=3 (prime), n=1024 int32 in [-1000, 1000], k = 2, 3, 4
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("k", [2, 3, 4])
def test_prime3_int32_exact(k):
    w = synth.WORKLOADS["prime3"]
    P, n = 3, w["n"]
    x = synth.host_ranks(w["seed"], P, n, np.int32, w["dist"])
    note("prime3 P=3 n=%d k=%d" % (n, k))
    for path in ([ar.AR_PATH_STEPWISE, ar.AR_PATH_FUSED] if k == 2 else [ar.AR_PATH_STEPWISE]):
        X = torch.from_numpy(x).to(DEV)
        run_plan(P, n, "int32", "sum", k, X, path)
        got = X.cpu().numpy()
        assert np.array_equal(got, oracle.allreduce(x, k, "sum"))
        assert np.array_equal(got, np.broadcast_to(oracle.direct(x, "sum"), (P, n)))


# ---------------------------------------------------------------------------
# Sweeps
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P", range(2, 17))
def test_tag_brute_force(P):
    """Rank x adds 1 << x: any missed or doubled term shows."""
    for k in ks(P):
        for n in (P - 1, 4 * P + 3, 1000):
            for path in paths(P, k):
                note("tags P=%d k=%d n=%d path=%d" % (P, k, n, path))
                x = np.stack([np.full(n, 1 << y, np.int32) for y in range(P)])
                X = torch.from_numpy(x).to(DEV)
                run_plan(P, n, "int32", "sum", k, X, path)
                assert np.all(X.cpu().numpy() == (1 << P) - 1), (P, k, n, path)


@pytest.mark.parametrize("P", range(2, 129))
def test_fp32_every_P_every_k(P):
    rng = np.random.default_rng(P)
    n = 3 * P + 5
    x = (rng.normal(size=(P, n)) * np.exp2(rng.integers(-6, 6, size=(P, n)))).astype(np.float32)
    for k in ks(P):
        want = oracle.allreduce(x, k, "sum")
        for path in paths(P, k):
            note("fp32 P=%d k=%d n=%d path=%d" % (P, k, n, path))
            X = torch.from_numpy(x).to(DEV)
            run_plan(P, n, "float32", "sum", k, X, path)
            got = X.cpu().numpy()
            assert np.array_equal(bits(got), bits(want)), (P, k, path)
            assert_fp32_bound(got, x)


@pytest.mark.parametrize("P,n", [(3, 100003), (5, 50001), (7, 65543), (24, 99991), (37, 74000), (64, 131072),
                                 (127, 130049)])
def test_several_tiles_per_block(P, n):
    """Blocks span several 1024-element tiles, with a ragged tail and blocks
    that start at every 16-byte phase."""
    rng = np.random.default_rng(n)
    x = rng.uniform(-1, 1, size=(P, n)).astype(np.float32)
    for k in sorted({ks(P)[0], ks(P)[len(ks(P)) // 2], ks(P)[-1]}):
        cols = sample_cols(n, P, per_block=96, seed=k)
        want = oracle.allreduce(np.ascontiguousarray(x[:, cols]), k, "sum", n=n, cols=cols)
        for path in paths(P, k):
            note("tiles P=%d n=%d k=%d path=%d" % (P, n, k, path))
            X = torch.from_numpy(x).to(DEV)
            run_plan(P, n, "float32", "sum", k, X, path)
            got = X.cpu().numpy()
            assert np.array_equal(bits(got[:, cols]), bits(want)), path
            assert_fp32_bound(got, x)


@pytest.mark.parametrize("P", [2, 3, 6, 13, 37, 100])
def test_max_exact(P):
    rng = np.random.default_rng(50 + P)
    n = 5 * P + 7
    xi = rng.integers(-2**31, 2**31, size=(P, n), dtype=np.int64).astype(np.int32)
    xf = rng.normal(size=(P, n)).astype(np.float32)
    xf[0, :3] = -0.0
    xf[1 % P, :3] = 0.0
    for k in ks(P):
        for path in paths(P, k):
            note("max P=%d k=%d path=%d" % (P, k, path))
            Xi = torch.from_numpy(xi).to(DEV)
            run_plan(P, n, "int32", "max", k, Xi, path)
            assert np.array_equal(Xi.cpu().numpy(), oracle.allreduce(xi, k, "max"))
            Xf = torch.from_numpy(xf).to(DEV)
            run_plan(P, n, "float32", "max", k, Xf, path)
            assert np.array_equal(bits(Xf.cpu().numpy()), bits(oracle.allreduce(xf, k, "max")))
            Xs = torch.from_numpy(xi).to(DEV)
            run_plan(P, n, "int32", "sum", k, Xs, path)
            assert np.array_equal(Xs.cpu().numpy(), oracle.allreduce(xi, k, "sum"))


# ---------------------------------------------------------------------------
# Edge cases
# ---------------------------------------------------------------------------

def test_degenerate_sizes():
    rng = np.random.default_rng(9)
    for P, n in [(5, 0), (5, 1), (5, 3), (37, 36), (2, 1), (2, 2), (2, 7), (1, 10)]:
        for k in ks(P):
            x = rng.normal(size=(P, n)).astype(np.float32)
            for path in paths(P, k):
                note("degenerate P=%d n=%d k=%d path=%d" % (P, n, k, path))
                X = torch.from_numpy(x).to(DEV)
                run_plan(P, n, "float32", "sum", k, X, path)
                assert np.array_equal(bits(X.cpu().numpy()), bits(oracle.allreduce(x, k, "sum"))), (P, n, k, path)


@pytest.mark.parametrize("shift", [1, 2, 3])
def test_unaligned_rank_buffers(shift):
    """4-byte aligned but not 16-byte aligned buffers take the scalar path."""
    rng = np.random.default_rng(shift)
    for P, n in [(7, 4099), (24, 2500)]:
        x = rng.normal(size=(P, n)).astype(np.float32)
        big = torch.zeros(P, n + 8, dtype=torch.float32, device=DEV)
        views = []
        for i in range(P):
            s = shift if i % 2 else 0
            big[i, s:s + n] = torch.from_numpy(x[i]).to(DEV)
            views.append(big[i, s:s + n])
        for k in ks(P):
            for path in paths(P, k):
                note("unaligned P=%d n=%d k=%d shift=%d path=%d" % (P, n, k, shift, path))
                for i in range(P):
                    s = shift if i % 2 else 0
                    big[i, s:s + n] = torch.from_numpy(x[i]).to(DEV)
                plan = ar.Plan(P, n, "float32", "sum", k, path=path)
                plan(views)
                torch.cuda.synchronize()
                got = np.stack([v.cpu().numpy() for v in views])
                assert np.array_equal(bits(got), bits(oracle.allreduce(x, k, "sum"))), (P, n, k, path)


def test_separate_allocations_and_shuffled_order():
    """Rank buffers need not be rows of one tensor nor in address order."""
    rng = np.random.default_rng(11)
    P, n, k = 13, 5003, 6
    x = rng.normal(size=(P, n)).astype(np.float32)
    ts = [torch.from_numpy(x[i]).to(DEV) for i in range(P)]
    pad = [torch.empty(1000, device=DEV) for _ in range(P)]  # noqa: F841 (spreads the addresses)
    plan = ar.Plan(P, n, "float32", "sum", k)
    note("separate allocations P=%d n=%d k=%d" % (P, n, k))
    plan(ts)
    torch.cuda.synchronize()
    got = np.stack([t.cpu().numpy() for t in ts])
    assert np.array_equal(bits(got), bits(oracle.allreduce(x, k, "sum")))


def test_aliasing_is_rejected_without_launch():
    P, n = 4, 100
    X = torch.zeros(P * n, device=DEV)
    plan = ar.Plan(P, n, "float32", "sum", 4)
    with pytest.raises(ar.ArError) as ei:
        plan([X[i * 50:] for i in range(P)])
    assert ei.value.status == ar.AR_ERR_ALIAS


# ---------------------------------------------------------------------------
# Batched instances, fused and step-wise paths
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("P", range(2, 17))
def test_fused_latency_optimal_matches_oracle_and_stepwise(P):
    rng = np.random.default_rng(300 + P)
    n, B = 37, 64
    L = ceil_log2(P)
    x = rng.normal(size=(P, B, n)).astype(np.float32)
    want = oracle.allreduce_batched(x, L, "sum")
    outs = {}
    for path in (ar.AR_PATH_FUSED, ar.AR_PATH_STEPWISE):
        note("batched LO P=%d n=%d B=%d path=%d" % (P, n, B, path))
        X = torch.from_numpy(x).to(DEV)
        plan = ar.Plan(P, n, "float32", "sum", L, path=path)
        plan.batched([X[i] for i in range(P)], B, n)
        torch.cuda.synchronize()
        outs[path] = X.cpu().numpy()
        assert np.array_equal(bits(outs[path]), bits(want)), path
    xi = rng.integers(-2**31, 2**31, size=(P, B, n), dtype=np.int64).astype(np.int32)
    for op in ("sum", "max"):
        X = torch.from_numpy(xi).to(DEV)
        plan = ar.Plan(P, n, "int32", op, L, path=ar.AR_PATH_FUSED)
        plan.batched([X[i] for i in range(P)], B, n)
        torch.cuda.synchronize()
        assert np.array_equal(X.cpu().numpy(), oracle.allreduce_batched(xi, L, op))


@pytest.mark.parametrize("P", [3, 5, 12, 16])
def test_fused_column_modes_agree(P, monkeypatch):
    """The fused latency-optimal kernel with and without nontemporal
    accesses produces the oracle's bits."""
    rng = np.random.default_rng(77 + P)
    n, B = 64, 40
    L = ceil_log2(P)
    x = rng.normal(size=(P, B, n)).astype(np.float32)
    want = oracle.allreduce_batched(x, L, "sum")
    for nt in ("0", "1"):
        monkeypatch.setenv("AR_FUSED_NT", nt)
        note("fused LO P=%d nt=%s" % (P, nt))
        X = torch.from_numpy(x).to(DEV)
        plan = ar.Plan(P, n, "float32", "sum", L, path=ar.AR_PATH_FUSED)
        plan.batched([X[i] for i in range(P)], B, n)
        torch.cuda.synchronize()
        assert np.array_equal(bits(X.cpu().numpy()), bits(want)), nt
    for nt in ("0", "1"):
        monkeypatch.setenv("AR_FUSED_NT", nt)
        note("fused BO nt=%s P=%d" % (nt, P))
        x2 = rng.normal(size=(P, 1001)).astype(np.float32)
        X = torch.from_numpy(x2).to(DEV)
        plan = ar.Plan(P, 1001, "float32", "sum", 2 * L, path=ar.AR_PATH_FUSED)
        plan([X[i] for i in range(P)])
        torch.cuda.synchronize()
        assert np.array_equal(bits(X.cpu().numpy()), bits(oracle.allreduce(x2, 2 * L, "sum"))), nt


@pytest.mark.parametrize("P,k", [(5, 3), (7, 4), (7, 6), (12, 6), (12, 8), (24, 10), (37, 8), (37, 12)])
def test_batched_with_gaps_leaves_gaps_untouched(P, k):
    rng = np.random.default_rng(P * 31 + k)
    n, B, stride = 53, 9, 61
    x = rng.normal(size=(P, B, stride)).astype(np.float32)
    want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), k, "sum")
    for path in paths(P, k):
        X = torch.from_numpy(x).to(DEV)
        note("batched gaps P=%d k=%d path=%d" % (P, k, path))
        plan = ar.Plan(P, n, "float32", "sum", k, path=path)
        plan.batched([X[i] for i in range(P)], B, stride)
        torch.cuda.synchronize()
        got = X.cpu().numpy()
        assert np.array_equal(bits(got[:, :, :n]), bits(want)), path
        assert np.array_equal(bits(got[:, :, n:]), bits(x[:, :, n:])), path


def test_small_batch_workload_full_size():
    """P in {5, 6, 7, 12}, n = 106 fp32 N(0,1), 65536 instances, k = ceil(log2 P):
    the fused kernel on all instances; the oracle on 512 sampled instances;
    the step-wise path on all instances for P = 5 (bit-identical)."""
    w = synth.WORKLOADS["small_batch"]
    n, B = w["n"], w["batch"]
    for P in w["P"]:
        L = ceil_log2(P)
        note("small_batch P=%d n=%d B=%d k=%d" % (P, n, B, L))
        X = synth.device_ranks(w["seed"], P, B * n, np.float32, w["dist"], DEV)
        X0 = X.clone() if P == 5 else None
        idx = np.sort(np.random.default_rng(P).choice(B, size=512, replace=False))
        xs = X.view(P, B, n)[:, torch.from_numpy(idx).to(DEV)].cpu().numpy()
        plan = ar.Plan(P, n, "float32", "sum", L)
        assert plan.stats().fused_ok == 1
        plan.batched([X[i] for i in range(P)], B, n)
        torch.cuda.synchronize()
        got = X.view(P, B, n)[:, torch.from_numpy(idx).to(DEV)].cpu().numpy()
        assert np.array_equal(bits(got), bits(oracle.allreduce_batched(xs, L, "sum")))
        for j in range(0, 512, 64):
            assert_fp32_bound(got[:, j], xs[:, j])
        if X0 is not None:
            ps = ar.Plan(P, n, "float32", "sum", L, path=ar.AR_PATH_STEPWISE)
            ps.batched([X0[i] for i in range(P)], B, n)
            torch.cuda.synchronize()
            assert torch.equal(X0.view(torch.int32), X.view(torch.int32))
        del X, X0
        torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# Full-size workloads, sampled columns
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("k", [11, 14, 7])
def test_medium127_workload_full_size(k):
    """P = 127, n = 2304 fp32 (9 KB), 8192 instances: the rank-slot kernel
    (k = 11 shifted; k = 14 bandwidth-optimal, split into the reducing launch
    and the broadcast) and the latency-optimal flat kernel (k = 7) on all
    instances; the oracle on 128 sampled instances."""
    w = synth.WORKLOADS["medium127"]
    P, n, B = 127, w["n"], w["batch"]
    note("medium127 P=%d n=%d B=%d k=%d" % (P, n, B, k))
    X = synth.device_ranks(w["seed"], P, B * n, np.float32, w["dist"], DEV)
    idx = np.sort(np.random.default_rng(k).choice(B, size=128, replace=False))
    it = torch.from_numpy(idx).to(DEV)
    xs = X.view(P, B, n)[:, it].cpu().numpy()
    plan = ar.Plan(P, n, "float32", "sum", k)
    st = plan.stats()
    assert st.fused_flat == (1 if k > 7 else 0) and st.fused_launches == (2 if k == 14 else 1)
    plan.batched([X[i] for i in range(P)], B, n)
    torch.cuda.synchronize()
    got = X.view(P, B, n)[:, it].cpu().numpy()
    assert np.array_equal(bits(got), bits(oracle.allreduce_batched(xs, k, "sum")))
    for j in range(0, 128, 32):
        assert_fp32_bound(got[:, j], xs[:, j])
    plan.close()
    del X
    torch.cuda.empty_cache()


@pytest.mark.parametrize("group,k", [("xor", 14), ("xor", 10), ("cyclic", 14)])
def test_medium128_workload_full_size(group, k):
    """P = 128, n = 2304 fp32 (9 KB), 8192 instances: the XOR group's flat
    kernel (Recursive Halving at k = 14, split into the reducing launch and
    the broadcast; the hybrid at k = 10) and the rank-slot kernel (cyclic,
    k = 14, split) on all instances; the oracle on 96 sampled instances."""
    w = synth.WORKLOADS["medium128"]
    P, n, B = 128, w["n"], w["batch"]
    note("medium128 %s P=%d n=%d B=%d k=%d" % (group, P, n, B, k))
    X = synth.device_ranks(w["seed"], P, B * n, np.float32, w["dist"], DEV)
    idx = np.sort(np.random.default_rng(k).choice(B, size=96, replace=False))
    it = torch.from_numpy(idx).to(DEV)
    xs = X.view(P, B, n)[:, it].cpu().numpy()
    plan = ar.Plan(P, n, "float32", "sum", k, group=group)
    st = plan.stats()
    assert st.fused_flat == 1 and st.fused_launches == (2 if k == 14 else 1)
    plan.batched([X[i] for i in range(P)], B, n)
    torch.cuda.synchronize()
    got = X.view(P, B, n)[:, it].cpu().numpy()
    assert np.array_equal(bits(got), bits(oracle.allreduce_batched(xs, k, "sum", group=group)))
    plan.close()
    del X
    torch.cuda.empty_cache()


def check_full_size(name, P, n, k, op, seed, dist):
    note("%s P=%d n=%d k=%d op=%s: fill" % (name, P, n, k, op))
    X = synth.device_ranks(seed, P, n, np.float32, dist, DEV)
    cols = sample_cols(n, P, per_block=48, seed=k)
    ct = torch.from_numpy(cols).to(DEV)
    xs = X[:, ct].cpu().numpy()
    ref_max = X.amax(dim=0) if op == "max" else None
    want = oracle.allreduce(xs, k, op, n=n, cols=cols)
    X0 = X.clone() if len(paths(P, k)) > 1 else None
    results = []
    for path in paths(P, k):
        if path != ar.AR_PATH_STEPWISE:
            X.copy_(X0)
        note("%s P=%d n=%d k=%d op=%s path=%d: execute" % (name, P, n, k, op, path))
        plan = ar.Plan(P, n, "float32", op, k, path=path)
        plan([X[i] for i in range(P)])
        torch.cuda.synchronize()
        got = X[:, ct].cpu().numpy()
        assert np.array_equal(bits(got), bits(want)), path
        if op == "sum":
            assert_fp32_bound(got, xs)
            if k == 2 * ceil_log2(P):  # bandwidth-optimal: every rank holds the same bits
                for i in range(1, P):
                    assert torch.equal(X[0].view(torch.int32), X[i].view(torch.int32))
                results.append(X[0].clone())
        else:
            for i in range(P):
                assert torch.equal(X[i], ref_max)
        plan.close()
    if len(results) == 2:  # the whole vector, not only the sampled columns, agrees across paths
        assert torch.equal(results[0].view(torch.int32), results[1].view(torch.int32))
    del X, X0, results
    torch.cuda.empty_cache()


def test_gradsync_workload():
    w = synth.WORKLOADS["gradsync"]
    check_full_size("gradsync", 24, w["n"], 10, "sum", w["seed"], w["dist"])


@pytest.mark.parametrize("k", [6, 7, 8, 9, 10, 11, 12])
@pytest.mark.parametrize("op", ["sum", "max"])
def test_prime_sweep_workload(k, op):
    w = synth.WORKLOADS["prime_sweep"]
    check_full_size("prime_sweep", 37, w["n"], k, op, w["seed"], w["dist"])


@pytest.mark.parametrize("k", [14, 10])
def test_large_workload(k):
    w = synth.WORKLOADS["large"]
    check_full_size("large", 127, w["n"], k, "sum", w["seed"], w["dist"])


def test_large_workload_ring():
    """The Ring at the large shape (P = 127, n = 2^26, k = 252): the fused
    chain's reducing launch and the destination-major broadcast; sampled
    columns against the oracle's Ring replay, and every rank the same bits."""
    w = synth.WORKLOADS["large"]
    P, n, k = 127, w["n"], 2 * 126
    note("large ring P=%d n=%d k=%d: fill" % (P, n, k))
    X = synth.device_ranks(w["seed"], P, n, np.float32, w["dist"], DEV)
    cols = sample_cols(n, P, per_block=16, seed=k)
    ct = torch.from_numpy(cols).to(DEV)
    xs = X[:, ct].cpu().numpy()
    want = oracle.allreduce(xs, k, "sum", n=n, cols=cols, schedule="ring")
    plan = ar.Plan(P, n, "float32", "sum", k, schedule="ring")
    st = plan.stats()
    assert st.fused_launches == 2 and st.fused_bcast_stream == 1
    note("large ring P=%d n=%d k=%d: execute" % (P, n, k))
    plan([X[i] for i in range(P)])
    torch.cuda.synchronize()
    got = X[:, ct].cpu().numpy()
    assert np.array_equal(bits(got), bits(want))
    assert_fp32_bound(got, xs)
    for i in range(1, P):
        assert torch.equal(X[0].view(torch.int32), X[i].view(torch.int32))
    plan.close()
    del X
    torch.cuda.empty_cache()


@pytest.mark.parametrize("P,group", [(17, "cyclic"), (24, "cyclic"), (37, "cyclic"), (64, "cyclic"), (127, "cyclic"),
                                     (32, "xor"), (128, "xor")])
def test_latency_optimal_flat_columns_with_gaps(P, group):
    """Latency-optimal plans above P = 16 tile the flat columns of all
    instances (blocks of a 106-element message hold at most one element at
    P = 127): many small instances with gaps between them, and a ragged n."""
    L = ceil_log2(P)
    rng = np.random.default_rng(P * 13)
    for n, B, stride in ((106, 37, 113), (P + 3, 5, P + 9), (1, 70, 2)):
        x = rng.normal(size=(P, B, stride)).astype(np.float32)
        want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), L, "sum", group=group)
        for path in (ar.AR_PATH_FUSED, ar.AR_PATH_STEPWISE):
            note("flat LO P=%d %s n=%d B=%d path=%d" % (P, group, n, B, path))
            X = torch.from_numpy(x).to(DEV)
            plan = ar.Plan(P, n, "float32", "sum", L, path=path, group=group)
            plan.batched([X[i] for i in range(P)], B, stride)
            torch.cuda.synchronize()
            got = X.cpu().numpy()
            assert np.array_equal(bits(got[:, :, :n]), bits(want)), (n, path)
            assert np.array_equal(bits(got[:, :, n:]), bits(x[:, :, n:])), (n, path)
            plan.close()
