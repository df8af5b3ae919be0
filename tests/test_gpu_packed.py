"""Packed column tiles against blocked ones, on the GPU, through the C ABI.

When blocks are short (many small instances), a column-fused wave takes one
block of several instances instead of one block of one instance, so that
its lanes stay busy while the rank rotation, which depends on the block
only, stays uniform.  Every kind of column launch -- bandwidth-optimal
(single and split into reduce plus broadcast), shifted, the XOR group's
halving and hybrid schedules, the Ring -- must give the oracle's bits with
packed tiles (AR_FUSED_PACKED=1), with blocked tiles (=0) and by default,
on batches with gaps between instances, ragged last tile groups and blocks
of zero, one or a few elements, and must leave the gaps untouched.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar
from test_gpu_parity import DEV, bits, note

pytestmark = pytest.mark.gpu

# P, n, batch, instance stride, k, group, schedule, op
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
]


@pytest.mark.parametrize("P,n,B,stride,k,group,schedule,op", CASES)
def test_packed_and_blocked_tiles_agree_with_oracle(P, n, B, stride, k, group, schedule, op, monkeypatch):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    rng = np.random.default_rng(P * 1000 + n + k)
    x = rng.normal(size=(P, B, stride)).astype(np.float32)
    want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), k, op, group=group, schedule=schedule)
    if op == "max":
        assert np.array_equal(want, np.broadcast_to(x[:, :, :n].max(axis=0), want.shape))
    for mode in ("0", "1", None):
        if mode is None:
            monkeypatch.delenv("AR_FUSED_PACKED", raising=False)
        else:
            monkeypatch.setenv("AR_FUSED_PACKED", mode)
        note("packed=%s %s/%s P=%d n=%d B=%d k=%d op=%s" % (mode, group, schedule, P, n, B, k, op))
        plan = ar.Plan(P, n, "float32", op, k, path=ar.AR_PATH_FUSED, group=group, schedule=schedule)
        X = torch.from_numpy(x).to(DEV)
        plan.batched([X[i] for i in range(P)], B, stride)
        torch.cuda.synchronize()
        got = X.cpu().numpy()
        plan.close()
        assert np.array_equal(bits(got[:, :, :n]), bits(want)), mode
        assert np.array_equal(bits(got[:, :, n:]), bits(x[:, :, n:])), mode
