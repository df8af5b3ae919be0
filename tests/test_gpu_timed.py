"""ar_execute_timed on the GPU, through the C ABI.

The timed execute must run the same kernels as ar_execute_batched -- its
results are the oracle's bits -- and report one positive duration per
launch: the k step launches (or merged runs) of the step-wise path, the
one or two launches of the fused path.
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


S, F, A = ar.AR_PATH_STEPWISE, ar.AR_PATH_FUSED, ar.AR_PATH_AUTO
CASES = [
    # P, n, batch, k, path, group, schedule
    (7, 10007, 1, 5, S, "cyclic", "butterfly"),      # shifted, scratch, 5 step launches
    (7, 10007, 1, 5, F, "cyclic", "butterfly"),
    (12, 106, 64, 4, A, "cyclic", "butterfly"),      # latency-optimal kernel
    (24, 106, 64, 10, F, "cyclic", "butterfly"),     # rank slots
    (24, 106, 64, 10, S, "cyclic", "butterfly"),     # merged runs
    (127, 12700, 1, 14, F, "cyclic", "butterfly"),   # reduce plus broadcast: two launches
    (16, 4099, 2, 6, S, "xor", "butterfly"),
    (16, 4099, 2, 6, F, "xor", "butterfly"),
    (5, 333, 1, 8, S, "cyclic", "ring"),
    (1, 100, 1, 0, A, "cyclic", "butterfly"),        # nothing to launch
    (6, 0, 1, 3, A, "cyclic", "butterfly"),
]


@pytest.mark.parametrize("P,n,B,k,path,group,schedule", CASES)
def test_timed_execute_matches_oracle_and_counts_launches(P, n, B, k, path, group, schedule):
    note("timed P=%d n=%d B=%d k=%d path=%d %s/%s" % (P, n, B, k, path, group, schedule))
    x = np.random.default_rng(P * 1000 + k).normal(size=(P, B, n)).astype(np.float32)
    X = torch.from_numpy(x).to(DEV)
    plan = ar.Plan(P, n, "float32", "sum", k, path=path, group=group, schedule=schedule)
    st = plan.stats()
    ms = plan.timed([X[i] for i in range(P)], B, n)
    torch.cuda.synchronize()
    fused = path == F or (path == A and st.fused_ok)
    want_launches = 0 if (P == 1 or n == 0) else (st.fused_launches if fused else st.launches)
    assert len(ms) == want_launches, (ms, st.fused_launches, st.launches)
    assert all(m > 0 for m in ms), ms
    if n:
        want = oracle.allreduce_batched(x, k, "sum", group=group, schedule=schedule)
        assert np.array_equal(bits(X.cpu().numpy()), bits(want))
    plan.close()


def test_timed_and_untimed_executes_agree_in_time():
    """The durations add up to about the time of the untimed execute (each
    launch's events add a few microseconds)."""
    P, n, k = 24, 1 << 22, 10
    X = torch.randn(P, n, device=DEV)
    plan = ar.Plan(P, n, "float32", "sum", k, path=S)
    bufs = [X[i] for i in range(P)]
    for _ in range(3):
        plan(bufs)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        plan(bufs)
    e1.record()
    torch.cuda.synchronize()
    untimed = e0.elapsed_time(e1) / 5
    timed = min(sum(plan.timed(bufs)) for _ in range(5))
    assert 0.8 * untimed < timed < 1.25 * untimed + 0.05, (timed, untimed)
    plan.close()
