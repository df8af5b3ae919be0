"""Python view of the CPU oracle (``oracle/oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``.  The HIP library never uses it.

The oracle replays the generalized Allreduce schedule of Kolmakov & Zhang
(arXiv:2004.09362, Secs. 5-9) rank by rank on the CPU, and also gives the
plain definition of Allreduce (Sec. 1; Sec. 5.4, the per-element reduction
result) for comparison.  See the header of ``oracle.c`` for the readings it
takes where the paper is silent.

This module only marshals numpy arrays into the C functions; it holds none of
the method's arithmetic.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

I32_SUM, I32_MAX, F32_SUM, F32_MAX, TERM = 0, 1, 2, 3, 4
GROUP_CYCLIC, GROUP_XOR = 0, 1
SCHED_BUTTERFLY, SCHED_RING = 0, 1
MAX_STEPS = 16
MAXP = 128

_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile liboracle.so with gcc (plain C, no fast-math, no contraction)."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c99", "-O2", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
           "-Wall", "-Wextra", "-Wno-unused-parameter", "-o", tmp, _SRC]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


class Trace(ctypes.Structure):
    _fields_ = [
        ("P", ctypes.c_int32), ("L", ctypes.c_int32), ("k", ctypes.c_int32),
        ("r", ctypes.c_int32), ("w", ctypes.c_int32),
        ("rs_steps", ctypes.c_int32), ("ag_steps", ctypes.c_int32),
        ("step_peer", ctypes.c_int32 * MAX_STEPS),
        ("pulls", ctypes.c_int32 * MAX_STEPS),
        ("combines", ctypes.c_int32 * MAX_STEPS),
        ("recv_blocks", ((ctypes.c_uint64 * 2) * MAXP) * MAX_STEPS),
    ]


def _configure(L):
    """Declare the C signatures on a loaded oracle library."""
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.oracle_terms_new.restype = vp
    L.oracle_terms_new.argtypes = []
    L.oracle_terms_free.argtypes = [vp]
    L.oracle_terms_violations.restype = i64
    L.oracle_terms_violations.argtypes = [vp]
    L.oracle_terms_count.restype = i64
    L.oracle_terms_count.argtypes = [vp]
    L.oracle_terms_render.restype = i64
    L.oracle_terms_render.argtypes = [vp, i32, ctypes.c_char_p, i64]
    L.oracle_terms_mask.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_uint64)]
    L.oracle_terms_block.restype = i32
    L.oracle_terms_block.argtypes = [vp, i32]
    L.oracle_allreduce.restype = ctypes.c_int
    L.oracle_allreduce.argtypes = [i32, i64, i32, i32, vp, i64, vp, i64, vp, i64, vp, vp]
    L.oracle_allreduce_batched.restype = ctypes.c_int
    L.oracle_allreduce_batched.argtypes = [i32, i64, i32, i32, vp, vp, i64]
    L.oracle_allreduce_ex.restype = ctypes.c_int
    L.oracle_allreduce_ex.argtypes = [i32, i64, i32, i32, i32, i32, vp, i64, vp, i64, vp, i64, vp, vp]
    L.oracle_allreduce_batched_ex.restype = ctypes.c_int
    L.oracle_allreduce_batched_ex.argtypes = [i32, i64, i32, i32, i32, i32, vp, vp, i64]
    L.oracle_direct_sum_f64.restype = ctypes.c_int
    L.oracle_direct_sum_f64.argtypes = [i32, i64, vp, i64, vp]
    L.oracle_direct_i32.restype = ctypes.c_int
    L.oracle_direct_i32.argtypes = [i32, i64, i32, vp, i64, vp]
    L.oracle_direct_max_f32.restype = ctypes.c_int
    L.oracle_direct_max_f32.argtypes = [i32, i64, vp, i64, vp]
    L.oracle_trace_size.restype = i32
    if L.oracle_trace_size() != ctypes.sizeof(Trace):
        raise RuntimeError("oracle trace layout mismatch")
    return L


def lib():
    """The oracle library built from ``oracle.c`` (compiled on first use)."""
    global _lib
    with _lock:
        if _lib is None:
            build()
            _lib = _configure(ctypes.CDLL(_LIB))
    return _lib


def load_variant(path: str):
    """Load another build of the oracle source (used by the tests that check
    that planted mistakes are caught).  Pass the handle as ``lib_=``."""
    return _configure(ctypes.CDLL(path))


def kind_of(dtype, op: str) -> int:
    dt = np.dtype(dtype)
    if dt == np.int32:
        return I32_SUM if op == "sum" else I32_MAX
    if dt == np.float32:
        return F32_SUM if op == "sum" else F32_MAX
    raise ValueError("oracle supports int32 and float32")


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _codes(group, schedule):
    g = {"cyclic": GROUP_CYCLIC, "xor": GROUP_XOR, GROUP_CYCLIC: GROUP_CYCLIC, GROUP_XOR: GROUP_XOR}[group]
    s = {"butterfly": SCHED_BUTTERFLY, "ring": SCHED_RING,
         SCHED_BUTTERFLY: SCHED_BUTTERFLY, SCHED_RING: SCHED_RING}[schedule]
    return g, s


def allreduce(x: np.ndarray, k: int, op: str = "sum", n: int | None = None,
              cols: np.ndarray | None = None, trace: bool = False, lib_=None,
              group="cyclic", schedule="butterfly"):
    """Replay the schedule.  ``x`` is [P, ncols] (int32 or float32).

    ``cols`` (optional) gives the global column index of each of the ncols
    columns (strictly increasing, in [0, n)); without it the columns are the
    whole vector and n = ncols.  ``group`` is "cyclic" or "xor" (power-of-two
    P), ``schedule`` "butterfly" (k in [L, 2L]) or "ring" (cyclic group,
    k = 2(P-1)).  Returns the [P, ncols] results, and the trace when
    ``trace`` is set.
    """
    g, sc = _codes(group, schedule)
    x = np.ascontiguousarray(x)
    P, ncols = x.shape
    kind = kind_of(x.dtype, op)
    if cols is None:
        n = ncols if n is None else n
        if n != ncols:
            raise ValueError("without cols, ncols must equal n")
        cp = None
    else:
        cols = np.ascontiguousarray(cols, dtype=np.int64)
        if n is None:
            raise ValueError("n is required with cols")
        cp = _ptr(cols)
    out = np.empty_like(x)
    tr = Trace() if trace else None
    rc = (lib_ or lib()).oracle_allreduce_ex(P, n, k, kind, g, sc, _ptr(x), ncols, _ptr(out), ncols, cp, ncols,
                                             None, ctypes.byref(tr) if tr is not None else None)
    if rc != 0:
        raise ValueError("oracle_allreduce rejected P=%d n=%s k=%d group=%s schedule=%s" % (P, n, k, group, schedule))
    return (out, tr) if trace else out


def allreduce_batched(x: np.ndarray, k: int, op: str = "sum", group="cyclic", schedule="butterfly") -> np.ndarray:
    """Independent instances; ``x`` is [P, batch, n]."""
    g, sc = _codes(group, schedule)
    x = np.ascontiguousarray(x)
    P, batch, n = x.shape
    out = np.empty_like(x)
    rc = lib().oracle_allreduce_batched_ex(P, n, k, kind_of(x.dtype, op), g, sc, _ptr(x), _ptr(out), batch)
    if rc != 0:
        raise ValueError("oracle_allreduce_batched rejected P=%d n=%d k=%d" % (P, n, k))
    return out


def direct(x: np.ndarray, op: str = "sum") -> np.ndarray:
    """Plain definition: [P, ncols] -> [ncols].  fp32 sums come back in fp64."""
    x = np.ascontiguousarray(x)
    P, ncols = x.shape
    L = lib()
    if x.dtype == np.int32:
        out = np.empty(ncols, np.int32)
        rc = L.oracle_direct_i32(P, ncols, I32_SUM if op == "sum" else I32_MAX, _ptr(x), ncols, _ptr(out))
    elif x.dtype == np.float32 and op == "sum":
        out = np.empty(ncols, np.float64)
        rc = L.oracle_direct_sum_f64(P, ncols, _ptr(x), ncols, _ptr(out))
    elif x.dtype == np.float32 and op == "max":
        out = np.empty(ncols, np.float32)
        rc = L.oracle_direct_max_f32(P, ncols, _ptr(x), ncols, _ptr(out))
    else:
        raise ValueError("unsupported dtype/op")
    if rc != 0:
        raise ValueError("oracle direct reduction failed")
    return out


class Terms:
    """Symbolic replay: the reduction tree of every output value."""

    def __init__(self, P: int, k: int, n: int | None = None, lib_=None, group="cyclic", schedule="butterfly"):
        g, sc = _codes(group, schedule)
        self.P, self.k = P, k
        self.n = P if n is None else n
        self._lib = L = lib_ or lib()
        self._h = L.oracle_terms_new()
        if not self._h:
            raise MemoryError
        self.ids = np.empty((P, self.n), np.int32)
        self.trace = Trace()
        dummy = np.zeros((P, self.n), np.int32)
        rc = L.oracle_allreduce_ex(P, self.n, k, TERM, g, sc, _ptr(dummy), self.n, _ptr(self.ids), self.n, None,
                                   self.n, self._h, ctypes.byref(self.trace))
        if rc != 0:
            L.oracle_terms_free(self._h)
            self._h = None
            raise ValueError("oracle term replay rejected P=%d k=%d" % (P, k))

    def __del__(self):
        if getattr(self, "_h", None):
            self._lib.oracle_terms_free(self._h)
            self._h = None

    @property
    def violations(self) -> int:
        return int(self._lib.oracle_terms_violations(self._h))

    @property
    def n_nodes(self) -> int:
        return int(self._lib.oracle_terms_count(self._h))

    def render(self, node: int) -> str:
        cap = 1 << 16
        buf = ctypes.create_string_buffer(cap)
        r = self._lib.oracle_terms_render(self._h, int(node), buf, cap)
        if r < 0:
            raise RuntimeError("render buffer too small")
        return buf.value.decode()

    def ranks(self, node: int) -> set[int]:
        m = (ctypes.c_uint64 * 2)()
        self._lib.oracle_terms_mask(self._h, int(node), m)
        return {y for y in range(self.P) if (m[y >> 6] >> (y & 63)) & 1}

    def block(self, node: int) -> int:
        return int(self._lib.oracle_terms_block(self._h, int(node)))

    def tree(self, rank: int, col: int) -> str:
        return self.render(self.ids[rank, col])
