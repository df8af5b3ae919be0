"""ar_execute_noalloc against ar_execute_batched on the GPU, through the C
ABI: the same plans on the same seeded inputs must give the same bits (and
the oracle's), on two calls in a row whose second is smaller -- the
library's per-device scratch array keeps the first call's contents, which
must not leak into the second.  Covered: step-wise plans with shifted
starting sets (the ones that use scratch: r > 0), a fused plan (no
scratch), two plans sharing the array alternately on one stream, and a call
beyond the array's 64 MiB, which is refused with nothing enqueued."""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar, synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
LIMIT = 64 << 20


def note(msg):
    print("[gpu] " + msg, flush=True)
    sys.stdout.flush()


def bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint32)


def inputs(seed, P, count, dtype):
    dist = synth.Dist("randint", -1000, 1000) if dtype == "int32" else synth.Dist("normal", 0.0, 1.0)
    return synth.host_ranks(seed, P, count, np.dtype(dtype), dist)


def run_both(plan, x, batch, stride):
    """The same call through ar_execute_batched and ar_execute_noalloc, on
    copies of x; returns both results."""
    P = x.shape[0]
    A = torch.from_numpy(x).to(DEV)
    B = A.clone()
    plan.batched([A[i] for i in range(P)], batch, stride)
    plan.noalloc([B[i] for i in range(P)], batch, stride)
    torch.cuda.synchronize()
    return A.cpu().numpy(), B.cpu().numpy()


# P, n, k, dtype, op, path, first batch, second (smaller) n and batch
CASES = [
    (7, 1000, 5, "float32", "sum", ar.AR_PATH_STEPWISE, 6, 333, 1),
    (37, 4101, 8, "int32", "max", ar.AR_PATH_STEPWISE, 3, 1200, 2),
    (127, 2304, 10, "float32", "sum", ar.AR_PATH_STEPWISE, 4, 2304, 1),
    (32, 5000, 7, "float32", "sum", ar.AR_PATH_STEPWISE, 2, 640, 1),
    (12, 106, 4, "float32", "sum", ar.AR_PATH_FUSED, 64, 106, 8),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "P%d_k%d_%s_%s_path%d" % (c[0], c[2], c[3], c[4], c[5]))
def test_noalloc_matches_execute_batched_twice(case):
    P, n, k, dtype, op, path, B1, n2, B2 = case
    group = "xor" if P == 32 else "cyclic"
    for call, (nn, B) in enumerate(((n, B1), (n2, B2))):
        plan = ar.Plan(P, nn, dtype, op, k, path=path, group=group)
        st = plan.stats()
        if path == ar.AR_PATH_STEPWISE:
            assert st.r > 0 and st.workspace_bytes > 0  # the plan uses scratch
            assert 2 * P * (-(-((B - 1) * nn + nn) // 64) * 64) * 4 <= LIMIT
        x = inputs(synth.BASE_SEED + 900 + 10 * P + call, P, B * nn, dtype)
        note("noalloc P=%d n=%d k=%d %s %s batch=%d call %d" % (P, nn, k, dtype, op, B, call))
        ref, got = run_both(plan, x, B, nn)
        assert np.array_equal(bits(got), bits(ref)), (case, call)
        want = oracle.allreduce_batched(x.reshape(P, B, nn), k, op, group=group)
        assert np.array_equal(bits(got), bits(want.reshape(P, B * nn))), (case, call)
        plan.close()


def test_two_plans_share_the_array_alternately():
    """Calls of different plans on one stream, ordered: each must see only
    its own scratch contents."""
    specs = [(37, 3000, 9), (127, 1500, 12), (5, 20000, 4)]
    plans = [ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_STEPWISE) for P, n, k in specs]
    xs = [inputs(synth.BASE_SEED + 950 + i, P, n, "float32") for i, (P, n, k) in enumerate(specs)]
    Xs = [torch.from_numpy(x).to(DEV) for x in xs]
    for rnd in range(2):
        for i in (0, 1, 2, 1, 0):
            P = specs[i][0]
            Xs[i].copy_(torch.from_numpy(xs[i]))
            plans[i].noalloc([Xs[i][y] for y in range(P)], 1, specs[i][1])
            torch.cuda.synchronize()
            want = oracle.allreduce(xs[i], specs[i][2], "sum")
            assert np.array_equal(bits(Xs[i].cpu().numpy()), bits(want)), (rnd, i)
    for p in plans:
        p.close()


def test_beyond_the_array_is_refused():
    P, n, k = 127, 70000, 10  # 2 * 127 * 70016 * 4 bytes > 64 MiB
    plan = ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_STEPWISE)
    X = torch.ones(P, n, device=DEV)
    with pytest.raises(ar.ArError) as ei:
        plan.noalloc([X[i] for i in range(P)], 1, n)
    assert ei.value.status == ar.AR_ERR_UNSUPPORTED and "at most" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((X == 1).all())  # nothing ran
    plan.close()


def test_noalloc_under_graph_capture():
    """The use it exists for: a step-wise plan with scratch captured into a
    graph with no allocation before or during the capture (one eager call
    looks up the device array first), replayed on fresh inputs."""
    P, n, k = 37, 2000, 8
    rng = np.random.default_rng(5150)
    plan = ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_STEPWISE)
    X = torch.empty((P, n), dtype=torch.float32, device=DEV)
    bufs = [X[i] for i in range(P)]
    x = rng.normal(size=(P, n)).astype(np.float32)
    X.copy_(torch.from_numpy(x))
    plan.noalloc(bufs, 1, n)
    torch.cuda.synchronize()
    assert np.array_equal(bits(X.cpu().numpy()), bits(oracle.allreduce(x, k, "sum")))
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            plan.noalloc(bufs, 1, n)
    torch.cuda.synchronize()
    for rep in range(3):
        x = rng.normal(size=(P, n)).astype(np.float32)
        X.copy_(torch.from_numpy(x))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits(X.cpu().numpy()), bits(oracle.allreduce(x, k, "sum"))), rep
    del g
    plan.close()
