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
import weakref
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

AR_K_AUTO = -1

EXPORTS = [
    "ar_plan_create", "ar_plan_create_ex", "ar_plan_set_path", "ar_execute", "ar_execute_batched", "ar_plan_stats",
    "ar_plan_num_launches", "ar_plan_launch", "ar_plan_destroy", "ar_status_string", "ar_last_error",
    "ar_last_error_message", "ar_model_time", "ar_model_best_k", "ar_plan_model_time", "ar_execute_timed",
    "ar_plan_dump", "ar_model_default_params", "ar_plan_model_seconds", "ar_plan_create_auto",
    "ar_execute_noalloc",
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
        ("fused_flat", ctypes.c_int32), ("exec_path", ctypes.c_int32), ("hbm_bytes_algorithmic", ctypes.c_int64),
        ("fused_bcast_stream", ctypes.c_int32),
    ]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class ModelParams(ctypes.Structure):
    """ar_model_params: the per-launch cost and HBM bandwidth of each path."""
    _fields_ = [("step_alpha", ctypes.c_double), ("step_bytes_per_s", ctypes.c_double),
                ("fused_alpha", ctypes.c_double), ("fused_bytes_per_s", ctypes.c_double)]

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
    L.ar_execute_noalloc.argtypes = [vp, ctypes.POINTER(vp), i64, i64, vp]
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
    L.ar_last_error_message.argtypes = []
    L.ar_last_error_message.restype = ctypes.c_char_p
    L.ar_model_default_params.argtypes = [ctypes.POINTER(ModelParams)]
    L.ar_plan_model_seconds.argtypes = [vp, ctypes.POINTER(ModelParams), i64, ctypes.c_int, ctypes.POINTER(dbl)]
    L.ar_plan_create_auto.argtypes = [i32, i64, ctypes.c_int, ctypes.c_int, ctypes.c_int, i64, ctypes.c_int,
                                      ctypes.POINTER(ModelParams), ctypes.POINTER(vp)]
    for name in ("ar_plan_create", "ar_plan_create_ex", "ar_plan_set_path", "ar_execute", "ar_execute_batched", "ar_plan_stats",
                 "ar_plan_num_launches", "ar_plan_launch", "ar_model_time", "ar_model_best_k", "ar_plan_model_time",
                 "ar_plan_dump", "ar_execute_timed", "ar_model_default_params", "ar_plan_model_seconds",
                 "ar_plan_create_auto", "ar_execute_noalloc"):
        getattr(L, name).restype = ctypes.c_int
    return L


lib = _load()


def status_name(s: int) -> str:
    return lib.ar_status_string(int(s)).decode()


def ar_last_error() -> str:
    return lib.ar_last_error().decode()


def ar_last_error_message() -> str:
    return lib.ar_last_error_message().decode()


def ar_status_string(s: int) -> str:
    return status_name(s)


def _check(st: int, where: str):
    if st != AR_OK:
        raise ArError(st, where, ar_last_error_message())


def _dtype_code(dtype) -> int:
    if dtype in (torch.int32, "int32", AR_INT32):
        return AR_INT32
    if dtype in (torch.float32, "float32", AR_FLOAT32):
        return AR_FLOAT32
    raise ArError(AR_ERR_UNSUPPORTED, "dtype", "int32 or float32 only, got %r" % (dtype,))


def _op_code(op) -> int:
    return {"sum": AR_SUM, "max": AR_MAX, AR_SUM: AR_SUM, AR_MAX: AR_MAX}[op]


# What the binding checks rank buffers against before a call reaches the
# library: P, n and dtype of each plan it created, by handle.
_PLAN_INFO: dict = {}


def _register(h: int, P: int, n: int, dtype_code: int) -> int:
    _PLAN_INFO[h] = (P, n, dtype_code)
    return h


def ar_plan_create(P: int, n: int, dtype, op, k_steps: int) -> int:
    h = ctypes.c_void_p()
    dt = _dtype_code(dtype)
    _check(lib.ar_plan_create(P, n, dt, _op_code(op), k_steps, ctypes.byref(h)), "ar_plan_create")
    return _register(h.value, P, n, dt)


def _group_code(group) -> int:
    return {"cyclic": AR_GROUP_CYCLIC, "xor": AR_GROUP_XOR, AR_GROUP_CYCLIC: AR_GROUP_CYCLIC,
            AR_GROUP_XOR: AR_GROUP_XOR}[group]


def _schedule_code(schedule) -> int:
    return {"butterfly": AR_SCHEDULE_BUTTERFLY, "ring": AR_SCHEDULE_RING, AR_SCHEDULE_BUTTERFLY: AR_SCHEDULE_BUTTERFLY,
            AR_SCHEDULE_RING: AR_SCHEDULE_RING}[schedule]


def ar_plan_create_ex(P: int, n: int, dtype, op, k_steps: int, group="cyclic", schedule="butterfly") -> int:
    h = ctypes.c_void_p()
    dt = _dtype_code(dtype)
    _check(lib.ar_plan_create_ex(P, n, dt, _op_code(op), k_steps, _group_code(group),
                                 _schedule_code(schedule), ctypes.byref(h)), "ar_plan_create_ex")
    return _register(h.value, P, n, dt)


def ar_model_default_params() -> ModelParams:
    mp = ModelParams()
    _check(lib.ar_model_default_params(ctypes.byref(mp)), "ar_model_default_params")
    return mp


def _params(params):
    """None, a ModelParams, or a dict with its four fields."""
    if params is None:
        return None
    if isinstance(params, ModelParams):
        return ctypes.byref(params)
    mp = ar_model_default_params()
    for key, val in dict(params).items():
        if key not in dict(ModelParams._fields_):
            raise KeyError("unknown model parameter %r" % key)
        setattr(mp, key, float(val))
    return ctypes.byref(mp)


def ar_plan_create_auto(P: int, n: int, dtype, op, group="cyclic", batch: int = 1, path: int = AR_PATH_AUTO,
                        params=None) -> int:
    h = ctypes.c_void_p()
    dt = _dtype_code(dtype)
    _check(lib.ar_plan_create_auto(P, n, dt, _op_code(op), _group_code(group), batch, int(path), _params(params),
                                   ctypes.byref(h)), "ar_plan_create_auto")
    return _register(h.value, P, n, dt)


def ar_plan_model_seconds(plan: int, params=None, batch: int = 1, path: int = AR_PATH_AUTO) -> float:
    t = ctypes.c_double()
    _check(lib.ar_plan_model_seconds(plan, _params(params), batch, int(path), ctypes.byref(t)),
           "ar_plan_model_seconds")
    return t.value


def ar_plan_set_path(plan: int, path: int):
    _check(lib.ar_plan_set_path(plan, int(path)), "ar_plan_set_path")


_TORCH_DTYPE = {AR_INT32: torch.int32, AR_FLOAT32: torch.float32}
# per plan: the last call whose buffers passed the checks (see _ptr_table)
_CHECKED: dict = {}


def _ptr_table(plan: int, rank_buffers, batch: int = 1, instance_stride: int | None = None,
               _on_gpu: bool = True) -> ctypes.Array:
    """The host table of rank pointers, after checking what the library
    cannot see: P entries, and for each torch tensor that it is contiguous,
    on the current GPU, of the plan's dtype, and that its storage holds the
    rank's (batch - 1) * instance_stride + n elements from the tensor's start.
    Raw integers are taken as device addresses, unchecked.  A failed check
    raises ArError(AR_ERR_INVALID_ARG) before anything is launched.
    (``_on_gpu=False`` skips the device checks so that the host tests can
    exercise the others on CPU tensors; every execute call keeps them.)"""
    bufs = list(rank_buffers)
    info = _PLAN_INFO.get(plan)
    if info is None:  # a handle this binding did not create
        st = ar_plan_stats(plan)
        info = _PLAN_INFO[plan] = (st.P, st.n, None)
    P, n, dt = info
    # the same (live) tensor objects at the same addresses as this plan's last
    # checked call -- what a loop of executes passes: only the addresses are
    # re-read (weak references, so the plan keeps no buffer alive)
    addrs = [b.data_ptr() if isinstance(b, torch.Tensor) else int(b) for b in bufs]
    key = (tuple(addrs), batch, instance_stride, _on_gpu)
    last = _CHECKED.get(plan)
    if last is not None and last[0] == key and len(last[1]) == len(bufs) and \
            all(r is None or r() is b for r, b in zip(last[1], bufs)):
        return (ctypes.c_void_p * P)(*addrs)
    if len(bufs) != P:
        raise ArError(AR_ERR_INVALID_ARG, "rank buffers", "the plan has P=%d ranks, got %d buffers" % (P, len(bufs)))
    if batch < 1:
        raise ArError(AR_ERR_INVALID_ARG, "rank buffers", "batch must be >= 1")
    stride = n if instance_stride is None or (batch == 1 and instance_stride < n) else instance_stride
    extent = (batch - 1) * stride + n if n > 0 else 0
    want = _TORCH_DTYPE.get(dt)
    dev = None
    storage_elems = {}
    for x, b in enumerate(bufs):
        if not isinstance(b, torch.Tensor):
            continue
        if extent > 0:
            if _on_gpu and not b.is_cuda:
                raise ArError(AR_ERR_INVALID_ARG, "rank buffers", "rank %d's tensor is not on a GPU" % x)
            if _on_gpu and dev is None:
                dev = torch.cuda.current_device()
            if _on_gpu and b.get_device() != dev:
                raise ArError(AR_ERR_INVALID_ARG, "rank buffers",
                              "rank %d's tensor is on cuda:%d, the current device is cuda:%d" % (x, b.get_device(), dev))
            if want is not None and b.dtype != want:
                raise ArError(AR_ERR_INVALID_ARG, "rank buffers",
                              "rank %d's tensor is %s, the plan's dtype is %s" % (x, b.dtype, want))
            if b.element_size() != 4 or not b.is_contiguous():
                raise ArError(AR_ERR_INVALID_ARG, "rank buffers",
                              "rank %d's tensor must be contiguous with 4-byte elements" % x)
            base = b._base if b._base is not None else b
            have = storage_elems.get(id(base))
            if have is None:
                have = storage_elems[id(base)] = base.untyped_storage().nbytes() // 4
            if have - b.storage_offset() < extent:
                raise ArError(AR_ERR_INVALID_ARG, "rank buffers",
                              "rank %d's tensor holds %d elements from its start, the call needs %d "
                              "((batch - 1) * instance_stride + n)" % (x, have - b.storage_offset(), extent))
    _CHECKED[plan] = (key, [weakref.ref(b) if isinstance(b, torch.Tensor) else None for b in bufs])
    return (ctypes.c_void_p * P)(*addrs)


def _stream_handle(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def ar_execute(plan: int, rank_buffers: Sequence, stream=None):
    tbl = _ptr_table(plan, rank_buffers)
    _check(lib.ar_execute(plan, tbl, _stream_handle(stream)), "ar_execute")


def ar_execute_batched(plan: int, rank_buffers: Sequence, batch: int, instance_stride: int, stream=None):
    tbl = _ptr_table(plan, rank_buffers, batch, instance_stride)
    _check(lib.ar_execute_batched(plan, tbl, batch, instance_stride, _stream_handle(stream)), "ar_execute_batched")


def ar_execute_noalloc(plan: int, rank_buffers: Sequence, batch: int, instance_stride: int, stream=None):
    """ar_execute_batched that never allocates device memory (scratch from
    the library's per-device array; see include/ar.h)."""
    tbl = _ptr_table(plan, rank_buffers, batch, instance_stride)
    _check(lib.ar_execute_noalloc(plan, tbl, batch, instance_stride, _stream_handle(stream)), "ar_execute_noalloc")


def ar_execute_timed(plan: int, rank_buffers: Sequence, batch: int = 1, instance_stride: int | None = None,
                     stream=None) -> list:
    """Execute, then wait for it; returns each launch's duration in ms."""
    st = ar_plan_stats(plan)
    stride = instance_stride if instance_stride is not None else st.n
    tbl = _ptr_table(plan, rank_buffers, batch, stride)
    cap = max(st.launches, st.fused_launches, 1)  # launches of either path
    ms = (ctypes.c_float * cap)()
    n = ctypes.c_int32()
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
    _PLAN_INFO.pop(plan, None)
    _CHECKED.pop(plan, None)
    lib.ar_plan_destroy(plan)


class Plan:
    """Owning handle around ``ar_plan*``.  ``k`` defaults to the
    bandwidth-optimal 2 ceil(log2 P) (the Ring: 2(P-1)); ``k="auto"`` (or
    AR_K_AUTO) lets the cost model choose k and, unless ``path`` fixes it,
    the path (ar_plan_create_auto, for ``batch`` instances per call)."""

    def __init__(self, P: int, n: int, dtype, op="sum", k=None, path: int = AR_PATH_AUTO,
                 group="cyclic", schedule="butterfly", batch: int = 1, params=None):
        L = max(0, (P - 1).bit_length())
        self.P, self.n = P, n
        self.handle = None
        ring = _schedule_code(schedule) == AR_SCHEDULE_RING
        if k in ("auto", AR_K_AUTO):
            if ring:
                raise ArError(AR_ERR_INVALID_ARG, "Plan", "the Ring has one step count, 2(P-1)")
            self.handle = ar_plan_create_auto(P, n, dtype, op, group, batch, path, params)
            self.k = ar_plan_stats(self.handle).k
            return
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

    def noalloc(self, rank_buffers, batch: int, instance_stride: int, stream=None):
        ar_execute_noalloc(self.handle, rank_buffers, batch, instance_stride, stream)

    def timed(self, rank_buffers, batch: int = 1, instance_stride: int | None = None, stream=None) -> list:
        """Execute and wait; the duration of each launch in milliseconds."""
        return ar_execute_timed(self.handle, rank_buffers, batch, instance_stride, stream)

    def dump(self) -> str:
        return ar_plan_dump(self.handle)

    def model_seconds(self, params=None, batch: int = 1, path: int = AR_PATH_AUTO) -> float:
        return ar_plan_model_seconds(self.handle, params, batch, path)

    def close(self):
        if self.handle:
            ar_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
