"""Performance floors on the GPU: catch a kernel that falls off its roofline.

Each case times a fused plan on two alternating input sets (so a launch does
not re-read what the previous one left in the 256 MB Infinity Cache) and
requires a loose fraction of the 8 TB/s HBM peak for the algorithmic bytes
(2 P n 4 per instance; (2P + 1) n 4 for a split launch).  Measured values are
65-82%; the floors sit well below them, so only a real regression -- a
kernel spilling registers, a launch shape gone wrong, a lost occupancy cap
-- trips them, not box-to-box variation.
"""
import pytest
import torch

from paper_2004_09362_amd import ar
from test_gpu_parity import DEV, note

pytestmark = pytest.mark.gpu

PEAK = 8000.0  # GB/s


def achieved(P, n, B, k, group, schedule, reps=10):
    plan = ar.Plan(P, n, "float32", "sum", k, path=ar.AR_PATH_FUSED, group=group, schedule=schedule)
    st = plan.stats()
    sets = [torch.randn(P, n * B, device=DEV) for _ in range(2)]
    tabs = [[X[i] for i in range(P)] for X in sets]
    for i in range(3):
        plan.batched(tabs[i & 1], B, n)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(reps):
        plan.batched(tabs[i & 1], B, n)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    plan.close()
    del sets, tabs
    torch.cuda.empty_cache()
    return st.hbm_bytes_fused * B / (ms * 1e-3) / 1e9


@pytest.mark.parametrize("name,P,n,B,k,group,schedule,floor", [
    ("latency-optimal P=12, 65536 x 106", 12, 106, 65536, 4, "cyclic", "butterfly", 0.55),
    ("latency-optimal P=127, 65536 x 106 (flat)", 127, 106, 65536, 7, "cyclic", "butterfly", 0.45),
    ("bandwidth-optimal P=24", 24, 1 << 23, 1, 10, "cyclic", "butterfly", 0.55),
    ("shifted P=37", 37, 1 << 22, 1, 8, "cyclic", "butterfly", 0.55),
    ("bandwidth-optimal P=127, split", 127, 1 << 23, 1, 14, "cyclic", "butterfly", 0.50),
    # the large workload's shape: 256 MiB rank buffers, the destination-major broadcast (measured 78-79%)
    ("bandwidth-optimal P=127, n=2^26, split, destination-major broadcast", 127, 1 << 26, 1, 14, "cyclic",
     "butterfly", 0.65),
    ("XOR Recursive Halving P=128, split", 128, 1 << 23, 1, 14, "xor", "butterfly", 0.50),
    ("XOR hybrid P=128", 128, 1 << 23, 1, 10, "xor", "butterfly", 0.50),
    ("Ring P=24", 24, 1 << 23, 1, 46, "cyclic", "ring", 0.55),
    # short blocks, rank slots on flat columns: 8192 messages of 9 KB at P = 127 (blocks of 18 elements),
    # measured 66% shifted (k = 11) and 80% split (k = 14, the Ring); the XOR group's Recursive Halving split
    # at P = 128, 79%; XOR and Ring batches of 4-5-element blocks, 70-79% and 65-70%
    ("shifted P=127, 8192 x 2304, rank slots", 127, 2304, 8192, 11, "cyclic", "butterfly", 0.55),
    ("bandwidth-optimal P=127, 8192 x 2304, rank slots, split", 127, 2304, 8192, 14, "cyclic", "butterfly", 0.6),
    ("Ring P=127, 8192 x 2304, rank slots, split", 127, 2304, 8192, 252, "cyclic", "ring", 0.6),
    ("XOR Recursive Halving P=128, 8192 x 2304, flat, split", 128, 2304, 8192, 14, "xor", "butterfly", 0.6),
    ("XOR P=32, 65536 x 128, flat", 32, 128, 65536, 10, "xor", "butterfly", 0.50),
    ("Ring P=24, 65536 x 106, rank slots", 24, 106, 65536, 46, "cyclic", "ring", 0.45),
])
def test_fused_kernels_stay_near_their_roofline(name, P, n, B, k, group, schedule, floor):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    gbs = achieved(P, n, B, k, group, schedule)
    note("perf %s: %.0f GB/s = %.1f%% of peak (floor %.0f%%)" % (name, gbs, 100 * gbs / PEAK, 100 * floor))
    assert gbs >= floor * PEAK, "%s: %.0f GB/s is below %.0f%% of the HBM peak" % (name, gbs, 100 * floor)
