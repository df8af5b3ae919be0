"""Stream ordering, concurrency and plan reuse on the GPU, through the C ABI.

An execute only enqueues work on the stream it is given (torch's current
stream by default), and a plan's scratch grows on the first execute that
needs more of it.  These tests run plans on side streams, two plans at once
on two streams, and one plan over batches that make its scratch grow and
then fit in it, each result against the oracle's bits.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar
from test_gpu_parity import DEV, bits, note

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu_present():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    yield


def _inputs(P, B, n, seed):
    return np.random.default_rng(seed).normal(size=(P, B, n)).astype(np.float32)


def test_two_plans_on_two_streams_at_once():
    """A shifted step-wise plan (scratch) and a fused plan, enqueued in turn on
    two side streams without synchronising in between, four rounds."""
    specs = [(7, 1001, 3, 5, ar.AR_PATH_STEPWISE), (37, 4000, 2, 9, ar.AR_PATH_FUSED)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    plans = [ar.Plan(P, n, "float32", "sum", k, path=path) for P, n, B, k, path in specs]
    rounds = []
    for rnd in range(4):
        xs, Xs = [], []
        for (P, n, B, k, path), s in zip(specs, streams):
            x = _inputs(P, B, n, 100 * rnd + P)
            with torch.cuda.stream(s):
                X = torch.from_numpy(x).to(DEV, non_blocking=False)
            xs.append(x)
            Xs.append(X)
        torch.cuda.synchronize()
        for plan, (P, n, B, k, path), s, X in zip(plans, specs, streams, Xs):
            note("streams round %d P=%d k=%d path=%d" % (rnd, P, k, path))
            plan.batched([X[i] for i in range(P)], B, n, s)
        rounds.append((xs, Xs))
    torch.cuda.synchronize()
    for xs, Xs in rounds:
        for (P, n, B, k, path), x, X in zip(specs, xs, Xs):
            assert np.array_equal(bits(X.cpu().numpy()), bits(oracle.allreduce_batched(x, k, "sum"))), (P, k)
    for p in plans:
        p.close()


@pytest.mark.parametrize("group,P,k", [("cyclic", 7, 5), ("cyclic", 24, 7), ("xor", 16, 6)])
def test_scratch_grows_with_the_batch(group, P, k):
    """One step-wise plan that needs scratch, run on a side stream on batches
    of 1, 9 (the scratch grows) and 4 (it fits) instances with gaps."""
    n = 3 * P + 2
    plan = ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_STEPWISE, group=group)
    assert plan.stats().workspace_bytes > 0
    s = torch.cuda.Stream()
    for B in (1, 9, 4):
        stride = n + 3
        x = _inputs(P, B, stride, 7 * B + P)
        want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), k, "sum", group=group)
        X = torch.from_numpy(x).to(DEV)
        torch.cuda.synchronize()
        note("scratch %s P=%d k=%d batch %d" % (group, P, k, B))
        plan.batched([X[i] for i in range(P)], B, stride, s)
        s.synchronize()
        got = X.cpu().numpy()
        assert np.array_equal(bits(got[:, :, :n]), bits(want)), B
        assert np.array_equal(bits(got[:, :, n:]), bits(x[:, :, n:])), B
    plan.close()


@pytest.mark.parametrize("path", [ar.AR_PATH_STEPWISE, ar.AR_PATH_FUSED])
def test_back_to_back_executes_of_one_plan(path):
    """Five executes of one plan on five input sets, enqueued back to back on
    one stream with no synchronisation: each set ends with its own result."""
    P, n, B, k = 13, 2000, 3, 6
    plan = ar.Plan(P, n, "float32", "sum", k, path=path)
    xs = [_inputs(P, B, n, 31 + i) for i in range(5)]
    Xs = [torch.from_numpy(x).to(DEV) for x in xs]
    torch.cuda.synchronize()
    for X in Xs:
        plan.batched([X[i] for i in range(P)], B, n)
    torch.cuda.synchronize()
    for x, X in zip(xs, Xs):
        assert np.array_equal(bits(X.cpu().numpy()), bits(oracle.allreduce_batched(x, k, "sum")))
    plan.close()
