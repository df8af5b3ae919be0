"""Seeded random plans under random combinations of the environment
overrides, against the CPU oracle.

Each case draws a group and schedule (cyclic butterfly, the XOR group, the
Ring), P, k, blocks of 0 to about 2100 elements, a batch with or without
gaps between instances, int32 or fp32, sum or max, the fused or the
step-wise path, rank rows on or off a 16-byte boundary, and a value (or
none) for each of AR_FUSED_ROTATE, AR_FUSED_SPLIT, AR_BCAST_STREAM,
AR_FUSED_PACKED, AR_BCAST_NT, AR_FUSED_CAP and AR_STEP_MERGE.  Whatever the
library makes of them, every result must carry the oracle's bits, and the
gaps and the padding around each rank's range must be left untouched.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar
from test_gpu_parity import DEV, bits, note

pytestmark = pytest.mark.gpu

OVERRIDES = {
    "AR_FUSED_ROTATE": [None, "0", "1"],
    "AR_FUSED_SPLIT": [None, "0", "1"],
    "AR_BCAST_STREAM": [None, "0", "1", "2", "3"],
    "AR_FUSED_PACKED": [None, "0", "1"],
    "AR_BCAST_NT": [None, "0", "1"],
    "AR_FUSED_CAP": [None, "0", "1", "3"],
    "AR_STEP_MERGE": [None, "0", "1"],
}
BLOCKS = [0, 1, 3, 17, 64, 65, 200, 1023, 1024, 1500, 2100]


def _cases(count, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        group = ["cyclic", "cyclic", "xor", "ring"][rng.integers(4)]
        P = int(2 ** rng.integers(1, 8)) if group == "xor" else int(rng.integers(2, 129))
        L = (P - 1).bit_length()
        if group == "ring":
            k, schedule, group = 2 * (P - 1), "ring", "cyclic"
        else:
            k, schedule = int(rng.integers(L, 2 * L + 1)), "butterfly"
        n = max(1, P * BLOCKS[rng.integers(len(BLOCKS))] + int(rng.integers(0, P)))
        B = min(int(rng.integers(1, 4)), max(1, 3_000_000 // (P * n)))
        stride = n if rng.integers(2) == 1 else n + int(rng.integers(1, 9))
        op = ["sum", "max"][rng.integers(2)]
        dtype = ["float32", "int32"][rng.integers(2)]
        path = [ar.AR_PATH_FUSED, ar.AR_PATH_FUSED, ar.AR_PATH_STEPWISE][rng.integers(3)]
        aligned = bool(rng.integers(2))
        env = tuple((v, c[rng.integers(len(c))]) for v, c in OVERRIDES.items())
        out.append((P, n, B, stride, k, group, schedule, op, dtype, path, aligned, env, int(rng.integers(1 << 30))))
    return out


@pytest.mark.parametrize("P,n,B,stride,k,group,schedule,op,dtype,path,aligned,env,seed", _cases(80, 20261206))
def test_random_plans_under_random_overrides(P, n, B, stride, k, group, schedule, op, dtype, path, aligned, env, seed,
                                             monkeypatch):
    for var, val in env:
        if val is None:
            monkeypatch.delenv(var, raising=False)
        else:
            monkeypatch.setenv(var, val)
    rng = np.random.default_rng(seed)
    if dtype == "int32":
        x = rng.integers(-2**31, 2**31, size=(P, B, stride), dtype=np.int64).astype(np.int32)
    else:
        x = rng.normal(size=(P, B, stride)).astype(np.float32)
    want = oracle.allreduce_batched(np.ascontiguousarray(x[:, :, :n]), k, op, group=group, schedule=schedule)
    span = (B - 1) * stride + n
    off = 0 if aligned else 1  # rank rows on a 16-byte boundary, or 4 bytes past one
    pitch = (span + 3) // 4 * 4 + 8
    big = torch.zeros(P, pitch, dtype=torch.float32 if dtype == "float32" else torch.int32, device=DEV)
    big[:, off:off + span] = torch.from_numpy(np.ascontiguousarray(x.reshape(P, B * stride)[:, :span])).to(DEV)
    note("sweep %s/%s P=%d n=%d B=%d stride=%d k=%d %s %s path=%d aligned=%d %s"
         % (group, schedule, P, n, B, stride, k, dtype, op, path, aligned, [e for e in env if e[1] is not None]))
    plan = ar.Plan(P, n, dtype, op, k, path=path, group=group, schedule=schedule)
    plan.batched([big[i, off:off + span] for i in range(P)], B, stride)
    torch.cuda.synchronize()
    h = big.cpu().numpy()
    plan.close()
    got = np.stack([h[:, off + j * stride:off + j * stride + n] for j in range(B)], axis=1)
    assert np.array_equal(bits(got), bits(want))
    for j in range(B - 1):  # the gaps between instances
        assert np.array_equal(bits(h[:, off + j * stride + n:off + (j + 1) * stride]), bits(x[:, j, n:stride]))
    assert not h[:, :off].any() and not h[:, off + span:].any()  # the padding around each rank's range
