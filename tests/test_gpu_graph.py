"""Executes captured into a HIP graph and replayed.

The library enqueues kernels only (no memset, no host synchronisation, no
allocation once the plan's scratch exists), so an execute that follows one
eager call on the same device and layout can be captured.  Each graph is
replayed several times on fresh inputs, with the program's own eager copies
and synchronisations in between, and every replay is checked bit for bit
against the CPU oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar
from test_gpu_parity import DEV, bits, note

pytestmark = pytest.mark.gpu

CASES = [
    # (P, n, batch, k, group, schedule, path)
    (7, 1001, 1, 5, "cyclic", "butterfly", ar.AR_PATH_STEPWISE),   # shifted: uses scratch
    (7, 1001, 1, 3, "cyclic", "butterfly", ar.AR_PATH_FUSED),
    (12, 106, 64, 4, "cyclic", "butterfly", ar.AR_PATH_FUSED),      # batched latency-optimal
    (8, 999, 1, 4, "xor", "butterfly", ar.AR_PATH_STEPWISE),       # XOR hybrid: scratch ping-pong
    (5, 777, 1, 8, "cyclic", "ring", ar.AR_PATH_STEPWISE),
    (24, 5000, 1, 10, "cyclic", "butterfly", ar.AR_PATH_STEPWISE),
]


def _capture_and_replay(P, n, B, k, group, schedule, path):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    rng = np.random.default_rng(P * 100 + k)
    note("graph P=%d n=%d B=%d k=%d %s/%s path=%d" % (P, n, B, k, group, schedule, path))
    plan = ar.Plan(P, n, "float32", "sum", k, path=path, group=group, schedule=schedule)
    X = torch.empty((P, B * n), dtype=torch.float32, device=DEV)
    bufs = [X[i] for i in range(P)]
    # eager call first: allocates the plan's scratch outside the capture
    X.copy_(torch.from_numpy(rng.normal(size=(P, B * n)).astype(np.float32)))
    plan.batched(bufs, B, n)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            plan.batched(bufs, B, n)
    torch.cuda.synchronize()
    for rep in range(3):
        x = rng.normal(size=(P, B, n)).astype(np.float32)
        X.copy_(torch.from_numpy(x.reshape(P, B * n)))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = X.cpu().numpy().reshape(P, B, n)
        want = oracle.allreduce_batched(x, k, "sum", group=group, schedule=schedule)
        assert np.array_equal(bits(got), bits(want)), rep
        # eager work between replays
        plan.batched(bufs, B, n)
        torch.cuda.synchronize()
    del g
    plan.close()


@pytest.mark.parametrize("P,n,B,k,group,schedule,path", CASES)
def test_captured_execute_replays_exactly(P, n, B, k, group, schedule, path):
    _capture_and_replay(P, n, B, k, group, schedule, path)


@pytest.mark.parametrize("P,n,B,k,group,rotate", [
    (127, 127 * 1024 + 76, 1, 14, "cyclic", "0"),   # block tiles (destination-major by the override)
    (127, 127 * 1024 + 76, 1, 14, "cyclic", None),  # the default rank slots below 256 MiB
    (127, 2304, 24, 14, "cyclic", None),            # flat columns, rank 0 holds the results
    (128, 2304, 16, 14, "xor", None),
])
def test_captured_split_with_the_destination_major_broadcast(P, n, B, k, group, rotate, monkeypatch):
    """The reducing launch and the destination-major broadcast captured
    together: replays on fresh inputs equal the oracle."""
    monkeypatch.setenv("AR_BCAST_STREAM", "1")
    if rotate is not None:
        monkeypatch.setenv("AR_FUSED_ROTATE", rotate)
    st = ar.Plan(P, n, "float32", "sum", k, group=group).stats()
    assert st.fused_launches == 2 and st.fused_bcast_stream == 1
    assert st.fused_flat == int(rotate is None)
    _capture_and_replay(P, n, B, k, group, "butterfly", ar.AR_PATH_FUSED)


def test_graph_stays_valid_when_the_scratch_grows():
    """A graph captured at batch 1 keeps working after an eager call with a
    larger batch made the plan allocate a larger scratch: the old buffer is
    kept until the plan is destroyed."""
    P, n, k = 7, 1001, 5
    rng = np.random.default_rng(4242)
    plan = ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_STEPWISE)
    assert plan.stats().workspace_bytes > 0
    X1 = torch.empty((P, n), dtype=torch.float32, device=DEV)
    b1 = [X1[i] for i in range(P)]
    X1.copy_(torch.from_numpy(rng.normal(size=(P, n)).astype(np.float32)))
    plan(b1)  # eager: scratch for batch 1
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            plan(b1)
    torch.cuda.synchronize()
    # eager call at batch 9: the plan's scratch grows
    B = 9
    x9 = rng.normal(size=(P, B, n)).astype(np.float32)
    X9 = torch.from_numpy(x9.reshape(P, B * n)).to(DEV)
    plan.batched([X9[i] for i in range(P)], B, n)
    torch.cuda.synchronize()
    assert np.array_equal(bits(X9.cpu().numpy().reshape(P, B, n)), bits(oracle.allreduce_batched(x9, k, "sum")))
    for rep in range(3):
        x = rng.normal(size=(P, n)).astype(np.float32)
        X1.copy_(torch.from_numpy(x))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits(X1.cpu().numpy()), bits(oracle.allreduce(x, k, "sum"))), rep
    del g
    plan.close()


def test_growth_under_capture_is_refused():
    """A captured call that would have to allocate more scratch is refused
    (nothing enqueued) instead of allocating inside the capture."""
    P, n, k = 7, 1001, 5
    plan = ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_STEPWISE)
    X1 = torch.ones((P, n), dtype=torch.float32, device=DEV)
    plan([X1[i] for i in range(P)])  # eager: scratch for batch 1
    torch.cuda.synchronize()
    B = 4
    X4 = torch.ones((P, B * n), dtype=torch.float32, device=DEV)
    Y = torch.ones(1024, device=DEV)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    status = None
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            try:
                plan.batched([X4[i] for i in range(P)], B, n)
            except ar.ArError as e:
                status = e.status
            Y.mul_(2.0)  # the capture holds this only
    torch.cuda.synchronize()
    assert status == ar.AR_ERR_UNSUPPORTED
    g.replay()
    torch.cuda.synchronize()
    assert bool((X4 == 1).all()) and bool((Y == 2).all())  # captured work runs only on replay
    del g
    plan.close()
