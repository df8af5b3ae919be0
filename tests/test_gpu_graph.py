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


@pytest.mark.parametrize("P,n,B,k,group,schedule,path", CASES)
def test_captured_execute_replays_exactly(P, n, B, k, group, schedule, path):
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
