"""Build libar.so (HIP kernels for gfx950 + host plan generator + C ABI).

Run ``python -m paper_2004_09362_amd.build`` or call :func:`build`.  Every
translation unit is compiled in parallel into ``_build/`` and linked into
``libar.so`` next to this file.
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libar.so")
SOURCES = [os.path.join(CSRC, f) for f in ["plan.cpp", "capi.cpp", "kernels.hip", "fused_lo.hip", "fused_group.hip",
                                           "broadcast.hip", "noalloc.hip"] +
           ["fused_col_g%d.hip" % i for i in range(8)]]
HEADERS = [os.path.join(CSRC, f) for f in ("ar_internal.hpp", "device_common.hpp", "fused_col.hpp")] + [
    os.path.join(ROOT, "include", "ar.h")]
OBJDIR = os.path.join(HERE, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
    # packed fp32 instructions stay off in all device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-ffp-contract=off", "-fno-fast-math",
    "-Wall", "-Wno-unused-function",
    "-I" + os.path.join(ROOT, "include"),
]


def _compile(src: str, incremental: bool = False) -> tuple[str, str]:
    obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
    if incremental and os.path.exists(obj):
        t = os.path.getmtime(obj)
        if all(os.path.getmtime(f) <= t for f in [src] + HEADERS):
            return obj, ""
    res = subprocess.run([HIPCC] + FLAGS + ["-c", src, "-o", obj], capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed on %s:\n%s%s" % (src, res.stdout, res.stderr))
    warn = [ln for ln in res.stderr.splitlines() if "packed-fp32-ops" not in ln and ln.strip()]
    return obj, "\n".join(warn)


def build(verbose: bool = False, incremental: bool = False) -> str:
    """Compile every source (in parallel) and link libar.so.  Rebuilds every
    unit unless ``incremental`` (then only units older than their sources)."""
    t0 = time.time()
    os.makedirs(OBJDIR, exist_ok=True)
    workers = max(1, min(len(SOURCES), int(os.environ.get("MAX_JOBS", os.cpu_count() or 1))))
    with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
        results = list(ex.map(lambda src: _compile(src, incremental), SOURCES))
    if verbose:
        for _, warn in results:
            if warn:
                sys.stderr.write(warn + "\n")
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=" + ARCH, "-o", tmp] + [o for o, _ in results]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("linking libar.so failed")
    os.replace(tmp, LIB)
    if verbose:
        print("built %s in %.1fs (%d units, %d parallel)" % (LIB, time.time() - t0, len(SOURCES), workers))
    return LIB


# Sources of each kernel family (besides the common ones): a profile taken on
# one family stays valid while only another family's sources change.
COMMON = ["capi.cpp", "ar_internal.hpp", "device_common.hpp"]
FAMILIES = {
    "step": ["kernels.hip", "plan.cpp", "noalloc.hip"],
    "lo": ["fused_lo.hip"],
    "col": ["fused_col.hpp"] + ["fused_col_g%d.hip" % i for i in range(8)],
    "group": ["fused_group.hip"],
    "bcast": ["broadcast.hip"],
}


def kernel_families(kernel: str) -> list[str]:
    """Families of a kernel name as bench.py reports it; a split launch
    ("<reducing kernel>+broadcast") has both kernels' families."""
    out = []
    for part in kernel.split("+"):
        for prefix, fam in (("step_kernel", "step"), ("fused_lo_kernel", "lo"), ("fused_bo_kernel", "col"),
                            ("fused_mid_kernel", "col"), ("fused_rot_kernel", "col"), ("fused_xor_kernel", "group"),
                            ("fused_ring_kernel", "group"), ("broadcast", "bcast")):
            if part.startswith(prefix):
                out.append(fam)
                break
        else:
            raise ValueError("unknown kernel %r" % kernel)
    return out


def code_text(text: str) -> str:
    """C++ source without comments and with whitespace collapsed: what the
    compiler sees, so that editing a comment does not count as a change."""
    import re

    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_hash(families) -> str:
    """Short hash of the code (comments removed) of one kernel family, or a
    list of families: counter profiles taken on other code are not reported
    as current."""
    import hashlib

    if isinstance(families, str):
        families = [families]
    h = hashlib.sha256()
    for f in COMMON + [f for fam in families for f in FAMILIES[fam]]:
        with open(os.path.join(CSRC, f), encoding="utf-8") as fh:
            h.update(f.encode())
            h.update(code_text(fh.read()).encode())
    return h.hexdigest()[:16]


def stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(f) > t for f in SOURCES + HEADERS)


if __name__ == "__main__":
    build(verbose=True, incremental="--incremental" in sys.argv)
