"""The Python binding refuses rank buffers that would make the library read
or write outside them, before any call reaches the library (no GPU needed):
a wrong number of buffers, tensors off the GPU, of the wrong dtype, not
contiguous, or whose storage ends before the call's extent."""
import os
import sys

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2004_09362_amd import ar  # noqa: E402


def _refused(fn, what):
    with pytest.raises(ar.ArError) as ei:
        fn()
    assert ei.value.status == ar.AR_ERR_INVALID_ARG
    assert what in str(ei.value)


def test_wrong_number_of_buffers():
    plan = ar.Plan(7, 100, "float32", "sum", 5)
    X = torch.zeros(7, 100)
    _refused(lambda: plan([X[i] for i in range(6)]), "P=7")
    _refused(lambda: plan.batched([X[i % 7] for i in range(8)], 1, 100), "P=7")
    _refused(lambda: ar._ptr_table(plan.handle, [X[i] for i in range(3)], _on_gpu=False), "got 3")


def test_cpu_tensors_are_refused_by_every_execute():
    plan = ar.Plan(5, 64, "float32", "sum", 3)
    X = torch.zeros(5, 64)
    bufs = [X[i] for i in range(5)]
    _refused(lambda: plan(bufs), "not on a GPU")
    _refused(lambda: plan.batched(bufs, 1, 64), "not on a GPU")
    _refused(lambda: plan.timed(bufs), "not on a GPU")


def test_dtype_contiguity_and_extent():
    P, n = 6, 50
    plan = ar.Plan(P, n, "int32", "max", 3)
    Xi = torch.zeros(P, 4 * n, dtype=torch.int32)
    tbl = ar._ptr_table(plan.handle, [Xi[i] for i in range(P)], 4, n, _on_gpu=False)
    assert len(tbl) == P and tbl[2] == Xi[2].data_ptr()
    Xf = torch.zeros(P, 4 * n, dtype=torch.float32)
    _refused(lambda: ar._ptr_table(plan.handle, [Xf[i] for i in range(P)], _on_gpu=False), "plan's dtype")
    Xt = torch.zeros(n, P, dtype=torch.int32)
    _refused(lambda: ar._ptr_table(plan.handle, [Xt[:, i] for i in range(P)], _on_gpu=False), "contiguous")
    # the last rank's storage ends 1 element short of (batch - 1) * stride + n
    _refused(lambda: ar._ptr_table(plan.handle, [Xi[i] for i in range(P - 1)] + [Xi.view(-1)[-(3 * 60 + n - 1):]],
                                   4, 60, _on_gpu=False), "needs %d" % (3 * 60 + n))
    # a row view may use the storage after it: the library checks overlaps between ranks itself
    ar._ptr_table(plan.handle, [Xi[i] for i in range(P)], 4, n, _on_gpu=False)
    # a batch of one takes n elements whatever the stride
    Xs = torch.zeros(P, n, dtype=torch.int32)
    ar._ptr_table(plan.handle, [Xs[i] for i in range(P)], 1, 7, _on_gpu=False)
    _refused(lambda: ar._ptr_table(plan.handle, [Xs[i] for i in range(P)], 0, n, _on_gpu=False), "batch")


def test_raw_addresses_and_empty_plans_pass_through():
    plan = ar.Plan(3, 0, "float32", "sum", 2)
    assert list(ar._ptr_table(plan.handle, [0, 0, 0])) == [None, None, None]
    plan([torch.zeros(1), torch.zeros(1), torch.zeros(1)], stream=0)  # n = 0: nothing is touched
    plan2 = ar.Plan(3, 10, "float32", "sum", 2)
    assert list(ar._ptr_table(plan2.handle, [4096, 8192, 12288])) == [4096, 8192, 12288]


def test_handles_created_elsewhere_are_checked_by_size():
    h = ar.lib  # a plan made through the raw C call, unknown to the binding's registry
    import ctypes
    p = ctypes.c_void_p()
    assert h.ar_plan_create(4, 40, ar.AR_FLOAT32, ar.AR_SUM, 3, ctypes.byref(p)) == ar.AR_OK
    try:
        _refused(lambda: ar._ptr_table(p.value, [torch.zeros(40)] * 3, _on_gpu=False), "P=4")
        X = torch.zeros(4, 40)
        ar._ptr_table(p.value, [X[i] for i in range(4)], _on_gpu=False)
    finally:
        ar.ar_plan_destroy(p.value)
