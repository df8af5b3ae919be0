"""Rank buffers of nearly 2^32 elements, on the GPU.

The destination-major broadcast indexes its column space in 32 bits and
takes batch * n up to 2^32 - 1 - 1024 (a chunk's last 16-byte group still
fits); the block-tiled column kernels count tiles in 32 bits; the fused
latency-optimal kernel and the step kernel walk columns in 64 bits.  These
cases sit just under 2^32 elements per rank at P = 2 (two 16 GiB rank
buffers): the latency-optimal plan in its fused kernel, the
bandwidth-optimal plan split into the reducing launch and the
destination-major broadcast (blocks off the 4 KB chunk grid, so boundary
chunks take two roots), and the bandwidth-optimal plan on the step-wise
path.  Sampled columns -- the first and last of every block, the last of
the buffer, random ones -- are compared with the oracle bit for bit, and for
the bandwidth-optimal plans the two ranks' whole vectors with each other.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2004_09362_amd import ar
from test_gpu_parity import DEV, bits, note, sample_cols

pytestmark = pytest.mark.gpu


def rows(P, n, seed):
    """[P, pitch] device tensor (pitch a multiple of 4, so every row starts
    on a 16-byte boundary), rows filled with N(0, 1) in their first n
    elements, and the row views of length n."""
    pitch = (n + 3) // 4 * 4
    X = torch.zeros((P, pitch), dtype=torch.float32, device=DEV)
    for x in range(P):
        g = torch.Generator(device=DEV)
        g.manual_seed(seed * 1000 + x)
        X[x, :n].normal_(0.0, 1.0, generator=g)
    return X, [X[x, :n] for x in range(P)]


@pytest.mark.parametrize("case", ["lo_fused", "split_stream", "stepwise"])
def test_columns_near_the_32_bit_limits(case, monkeypatch):
    P = 2
    if case == "lo_fused":
        n, k, path = (1 << 32) - 100, 1, ar.AR_PATH_FUSED
    elif case == "split_stream":
        n, k, path = (1 << 32) - 2046, 2, ar.AR_PATH_FUSED  # blocks of 2^31 - 1023: off the chunk grid
        monkeypatch.setenv("AR_FUSED_SPLIT", "1")
        monkeypatch.setenv("AR_BCAST_STREAM", "1")
    else:
        n, k, path = (1 << 32) - 100, 2, ar.AR_PATH_STEPWISE
    plan = ar.Plan(P, n, "float32", "sum", k, path=path)
    st = plan.stats()
    if case == "lo_fused":
        assert st.exec_path == ar.AR_PATH_FUSED
    if case == "split_stream":
        assert st.fused_launches == 2 and st.fused_bcast_stream == 1
    note("limits %s: P=%d n=%d k=%d path=%d: fill" % (case, P, n, k, path))
    X, views = rows(P, n, seed=n % 9973 + k)
    cols = np.unique(np.concatenate([sample_cols(n, P, per_block=64, seed=k), np.arange(n - 70, n)]))
    ct = torch.from_numpy(cols).to(DEV)
    xs = X[:, ct].cpu().numpy()
    want = oracle.allreduce(xs, k, "sum", n=n, cols=cols)
    note("limits %s: execute" % case)
    plan(views)
    torch.cuda.synchronize()
    got = X[:, ct].cpu().numpy()
    assert np.array_equal(bits(got), bits(want))
    if k == 2:  # bandwidth-optimal: both ranks hold the same bits everywhere
        assert torch.equal(X[0, :n].view(torch.int32), X[1, :n].view(torch.int32))
    assert not X[:, n:].any().item()  # the row padding is never written
    plan.close()
    del X, views
    torch.cuda.empty_cache()
