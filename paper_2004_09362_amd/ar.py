"""Thin Python binding of libar.so (``include/ar.h``).

Argument marshalling only: every function forwards to the C entry point of
the same name, and all arithmetic happens in the library's HIP kernels.
PyTorch is used for device memory and streams: rank buffers are torch
tensors (or raw device addresses), the stream is torch's current stream
unless one is given.  There is no fallback: if the built library is absent
the import fails, and on a machine without a GPU the execute calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

import torch  # noqa: F401  (loads the HIP runtime torch was built with, before libar.so)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libar.so")

AR_OK, AR_ERR_INVALID_ARG, AR_ERR_UNSUPPORTED, AR_ERR_ALIAS = 0, 1, 2, 3
AR_ERR_OUT_OF_MEMORY, AR_ERR_HIP, AR_ERR_NO_DEVICE, AR_ERR_INTERNAL = 4, 5, 6, 7
AR_INT32, AR_FLOAT32 = 0, 1
AR_SUM, AR_MAX = 0, 1
AR_PATH_AUTO, AR_PATH_STEPWISE, AR_PATH_FUSED = 0, 1, 2
AR_KIND_COPY, AR_KIND_REDUCE, AR_KIND_REDUCE2 = 0, 1, 2
AR_GROUP_CYCLIC, AR_GROUP_XOR = 0, 1
AR_SCHEDULE_BUTTERFLY, AR_SCHEDULE_RING = 0, 1

EXPORTS = [
    "ar_plan_create", "ar_plan_create_ex", "ar_plan_set_path", "ar_execute", "ar_execute_batched", "ar_plan_stats",
    "ar_plan_num_launches", "ar_plan_launch", "ar_plan_destroy", "ar_status_string", "ar_last_error",
    "ar_model_time", "ar_model_best_k", "ar_plan_model_time", "ar_execute_timed", "ar_plan_dump",
]


class ArError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__("%s: %s (%s)" % (where, detail, status_name(status)))
        self.status = status


class Stats(ctypes.Structure):
    _fields_ = [
        ("P", ctypes.c_int32), ("L", ctypes.c_int32), ("k", ctypes.c_int32), ("r", ctypes.c_int32),
        ("w", ctypes.c_int32), ("rs_steps", ctypes.c_int32), ("ag_steps", ctypes.c_int32),
        ("launches", ctypes.c_int32), ("fused_ok", ctypes.c_int32),
        ("n", ctypes.c_int64), ("elem_bytes", ctypes.c_int64),
        ("blocks_pulled_per_rank", ctypes.c_int64),
        ("bytes_pulled_per_rank_min", ctypes.c_int64), ("bytes_pulled_per_rank_max", ctypes.c_int64),
        ("bytes_pulled_total", ctypes.c_int64), ("combines_per_rank", ctypes.c_int64),
        ("hbm_bytes_stepwise", ctypes.c_int64), ("hbm_bytes_fused", ctypes.c_int64),
        ("workspace_bytes", ctypes.c_int64),
        ("group", ctypes.c_int32), ("schedule", ctypes.c_int32), ("fused_launches", ctypes.c_int32),
        ("fused_flat", ctypes.c_int32),
    ]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class LaunchDesc(ctypes.Structure):
    _fields_ = [("phase", ctypes.c_int32), ("n_ranges", ctypes.c_int32)]


class RangeDesc(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in
                ("p0", "count", "kind", "delta", "dst", "own", "dst2", "own2", "src")]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libar.so is not built (%s); run `python -m paper_2004_09362_amd.build`" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.ar_plan_create.argtypes = [i32, i64, ctypes.c_int, ctypes.c_int, i32, ctypes.POINTER(vp)]
    L.ar_plan_create_ex.argtypes = [i32, i64, ctypes.c_int, ctypes.c_int, i32, ctypes.c_int, ctypes.c_int,
                                    ctypes.POINTER(vp)]
    L.ar_plan_set_path.argtypes = [vp, ctypes.c_int]
    L.ar_execute.argtypes = [vp, ctypes.POINTER(vp), vp]
    L.ar_execute_batched.argtypes = [vp, ctypes.POINTER(vp), i64, i64, vp]
    L.ar_plan_stats.argtypes = [vp, ctypes.POINTER(Stats)]
    L.ar_plan_num_launches.argtypes = [vp, ctypes.POINTER(i32)]
    L.ar_plan_launch.argtypes = [vp, i32, ctypes.POINTER(LaunchDesc), ctypes.POINTER(RangeDesc), i32]
    L.ar_plan_dump.argtypes = [vp, ctypes.c_char_p, i64, ctypes.POINTER(i64)]
    L.ar_execute_timed.argtypes = [vp, ctypes.POINTER(vp), i64, i64, vp, ctypes.POINTER(ctypes.c_float), i32,
                                   ctypes.POINTER(i32)]
    L.ar_plan_destroy.argtypes = [vp]
    L.ar_plan_destroy.restype = None
    dbl = ctypes.c_double
    L.ar_model_time.argtypes = [i32, dbl, i32, dbl, dbl, dbl, ctypes.POINTER(dbl)]
    L.ar_model_best_k.argtypes = [i32, dbl, dbl, dbl, dbl, ctypes.POINTER(i32), ctypes.POINTER(dbl)]
    L.ar_plan_model_time.argtypes = [vp, dbl, dbl, dbl, ctypes.POINTER(dbl)]
    L.ar_status_string.argtypes = [ctypes.c_int]
    L.ar_status_string.restype = ctypes.c_char_p
    L.ar_last_error.argtypes = []
    L.ar_last_error.restype = ctypes.c_char_p
    for name in ("ar_plan_create", "ar_plan_create_ex", "ar_plan_set_path", "ar_execute", "ar_execute_batched", "ar_plan_stats",
                 "ar_plan_num_launches", "ar_plan_launch", "ar_model_time", "ar_model_best_k", "ar_plan_model_time",
                 "ar_plan_dump", "ar_execute_timed"):
        getattr(L, name).restype = ctypes.c_int
    return L


lib = _load()


def status_name(s: int) -> str:
    return lib.ar_status_string(int(s)).decode()


def ar_last_error() -> str:
    return lib.ar_last_error().decode()


def ar_status_string(s: int) -> str:
    return status_name(s)


def _check(st: int, where: str):
    if st != AR_OK:
        raise ArError(st, where, ar_last_error())


def _dtype_code(dtype) -> int:
    if dtype in (torch.int32, "int32", AR_INT32):
        return AR_INT32
    if dtype in (torch.float32, "float32", AR_FLOAT32):
        return AR_FLOAT32
    raise ArError(AR_ERR_UNSUPPORTED, "dtype", "int32 or float32 only, got %r" % (dtype,))


def _op_code(op) -> int:
    return {"sum": AR_SUM, "max": AR_MAX, AR_SUM: AR_SUM, AR_MAX: AR_MAX}[op]


def ar_plan_create(P: int, n: int, dtype, op, k_steps: int) -> int:
    h = ctypes.c_void_p()
    _check(lib.ar_plan_create(P, n, _dtype_code(dtype), _op_code(op), k_steps, ctypes.byref(h)), "ar_plan_create")
    return h.value


def _group_code(group) -> int:
    return {"cyclic": AR_GROUP_CYCLIC, "xor": AR_GROUP_XOR, AR_GROUP_CYCLIC: AR_GROUP_CYCLIC,
            AR_GROUP_XOR: AR_GROUP_XOR}[group]


def _schedule_code(schedule) -> int:
    return {"butterfly": AR_SCHEDULE_BUTTERFLY, "ring": AR_SCHEDULE_RING, AR_SCHEDULE_BUTTERFLY: AR_SCHEDULE_BUTTERFLY,
            AR_SCHEDULE_RING: AR_SCHEDULE_RING}[schedule]


def ar_plan_create_ex(P: int, n: int, dtype, op, k_steps: int, group="cyclic", schedule="butterfly") -> int:
    h = ctypes.c_void_p()
    _check(lib.ar_plan_create_ex(P, n, _dtype_code(dtype), _op_code(op), k_steps, _group_code(group),
                                 _schedule_code(schedule), ctypes.byref(h)), "ar_plan_create_ex")
    return h.value


def ar_plan_set_path(plan: int, path: int):
    _check(lib.ar_plan_set_path(plan, int(path)), "ar_plan_set_path")


def _ptr_table(rank_buffers) -> ctypes.Array:
    addrs = []
    for b in rank_buffers:
        addrs.append(b.data_ptr() if isinstance(b, torch.Tensor) else int(b))
    return (ctypes.c_void_p * len(addrs))(*addrs)


def _stream_handle(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def ar_execute(plan: int, rank_buffers: Sequence, stream=None):
    tbl = _ptr_table(rank_buffers)
    _check(lib.ar_execute(plan, tbl, _stream_handle(stream)), "ar_execute")


def ar_execute_batched(plan: int, rank_buffers: Sequence, batch: int, instance_stride: int, stream=None):
    tbl = _ptr_table(rank_buffers)
    _check(lib.ar_execute_batched(plan, tbl, batch, instance_stride, _stream_handle(stream)), "ar_execute_batched")


def ar_execute_timed(plan: int, rank_buffers: Sequence, batch: int = 1, instance_stride: int | None = None,
                     stream=None) -> list:
    """Execute, then wait for it; returns each launch's duration in ms."""
    tbl = _ptr_table(rank_buffers)
    st = ar_plan_stats(plan)
    cap = max(st.launches, st.fused_launches, 1)  # launches of either path
    ms = (ctypes.c_float * cap)()
    n = ctypes.c_int32()
    stride = instance_stride if instance_stride is not None else st.n
    _check(lib.ar_execute_timed(plan, tbl, batch, stride, _stream_handle(stream), ms, cap, ctypes.byref(n)),
           "ar_execute_timed")
    return list(ms[:min(n.value, cap)])


def ar_plan_dump(plan: int) -> str:
    n = ctypes.c_int64()
    _check(lib.ar_plan_dump(plan, None, 0, ctypes.byref(n)), "ar_plan_dump")
    buf = ctypes.create_string_buffer(n.value + 1)
    _check(lib.ar_plan_dump(plan, buf, n.value + 1, ctypes.byref(n)), "ar_plan_dump")
    return buf.value.decode()


def ar_plan_stats(plan: int) -> Stats:
    s = Stats()
    _check(lib.ar_plan_stats(plan, ctypes.byref(s)), "ar_plan_stats")
    return s


def ar_plan_num_launches(plan: int) -> int:
    v = ctypes.c_int32()
    _check(lib.ar_plan_num_launches(plan, ctypes.byref(v)), "ar_plan_num_launches")
    return v.value


def ar_plan_launch(plan: int, i: int):
    d = LaunchDesc()
    _check(lib.ar_plan_launch(plan, i, ctypes.byref(d), None, 0), "ar_plan_launch")
    rs = (RangeDesc * max(1, d.n_ranges))()
    _check(lib.ar_plan_launch(plan, i, ctypes.byref(d), rs, d.n_ranges), "ar_plan_launch")
    return d.phase, [rs[j].as_dict() for j in range(d.n_ranges)]


def ar_model_time(P: int, m_bytes: float, k_steps: int, alpha: float, beta: float, gamma: float) -> float:
    t = ctypes.c_double()
    _check(lib.ar_model_time(P, m_bytes, k_steps, alpha, beta, gamma, ctypes.byref(t)), "ar_model_time")
    return t.value


def ar_model_best_k(P: int, m_bytes: float, alpha: float, beta: float, gamma: float):
    k, r = ctypes.c_int32(), ctypes.c_double()
    _check(lib.ar_model_best_k(P, m_bytes, alpha, beta, gamma, ctypes.byref(k), ctypes.byref(r)), "ar_model_best_k")
    return k.value, r.value


def ar_plan_model_time(plan: int, alpha: float, beta: float, gamma: float) -> float:
    t = ctypes.c_double()
    _check(lib.ar_plan_model_time(plan, alpha, beta, gamma, ctypes.byref(t)), "ar_plan_model_time")
    return t.value


def ar_plan_destroy(plan: int):
    lib.ar_plan_destroy(plan)


class Plan:
    """Owning handle around ``ar_plan*``.  ``k`` defaults to the
    bandwidth-optimal 2 ceil(log2 P) (the Ring: 2(P-1))."""

    def __init__(self, P: int, n: int, dtype, op="sum", k: int | None = None, path: int = AR_PATH_AUTO,
                 group="cyclic", schedule="butterfly"):
        L = max(0, (P - 1).bit_length())
        self.P, self.n = P, n
        ring = _schedule_code(schedule) == AR_SCHEDULE_RING
        self.k = (2 * (P - 1) if ring else 2 * L) if k is None else k
        self.handle = ar_plan_create_ex(P, n, dtype, op, self.k, group, schedule)
        if path != AR_PATH_AUTO:
            ar_plan_set_path(self.handle, path)

    def set_path(self, path: int):
        ar_plan_set_path(self.handle, path)

    def stats(self) -> Stats:
        return ar_plan_stats(self.handle)

    def launches(self):
        return [ar_plan_launch(self.handle, i) for i in range(ar_plan_num_launches(self.handle))]

    def __call__(self, rank_buffers, stream=None):
        ar_execute(self.handle, rank_buffers, stream)

    def batched(self, rank_buffers, batch: int, instance_stride: int, stream=None):
        ar_execute_batched(self.handle, rank_buffers, batch, instance_stride, stream)

    def timed(self, rank_buffers, batch: int = 1, instance_stride: int | None = None, stream=None) -> list:
        """Execute and wait; the duration of each launch in milliseconds."""
        return ar_execute_timed(self.handle, rank_buffers, batch, instance_stride, stream)

    def dump(self) -> str:
        return ar_plan_dump(self.handle)

    def close(self):
        if self.handle:
            ar_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
