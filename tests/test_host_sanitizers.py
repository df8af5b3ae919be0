"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer.

Two drivers under tests/native/, compiled here with g++ / gcc -- host code
only; no HIP source is built with a sanitizer:

- host_sanitize.cpp links the library's plan generator and C ABI (plan.cpp,
  capi.cpp) against a fake one-device HIP runtime and launchers that check
  the arguments the kernels would receive.  It sweeps every P in 1..128 and
  every k, group and schedule over empty, tiny, ragged and large n; replays
  the launch tables on exactly sized host rows against the plain definition;
  and drives every error path: bad arguments, aliasing, sizes that would
  overflow, no device, failed scratch allocations and failed launches.
  LeakSanitizer and the fake allocator's count show that nothing leaks.
- oracle_sanitize.c links the CPU oracle alone.  It replays every schedule
  on exactly sized buffers and checks the results against the plain
  definition (bit for bit for integers and maxima, and within the
  summation-order error bound for fp32 sums), the column sampling, the
  batching and the term mode.

host_sanitize.cpp also runs on eight threads at once under ThreadSanitizer.
Either driver exits non-zero on a failed check, and a sanitizer report
aborts it (-fno-sanitize-recover, halt_on_error).
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2004_09362_amd", "csrc")
NATIVE = os.path.join(ROOT, "tests", "native")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(exe, *args, timeout=600):
    res = subprocess.run([str(exe), *map(str, args)], capture_output=True, text=True, timeout=timeout, env=ENV)
    return res.returncode, res.stdout + res.stderr


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ is not installed")
def test_library_host_code_under_sanitizers(tmp_path):
    if not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime_api.h")):
        pytest.skip("HIP headers not found")
    exe = tmp_path / "host_sanitize"
    subprocess.run(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"),
                    "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-o", str(exe),
                    os.path.join(NATIVE, "host_sanitize.cpp"), os.path.join(CSRC, "capi.cpp"),
                    os.path.join(CSRC, "plan.cpp"), "-pthread"], check=True)
    rc, out = _run(exe)
    assert rc == 0, out[-4000:]
    assert "0 launch contract problems, 0 failures" in out, out[-4000:]


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ is not installed")
def test_library_host_code_from_eight_threads_under_thread_sanitizer(tmp_path):
    """Plans created, dumped, timed and executed (fake runtime) on eight
    threads at once, with the error checks on a ninth: the error text is
    per thread and the device LDS sizes are cached in atomics, so
    ThreadSanitizer must find no race."""
    if not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime_api.h")):
        pytest.skip("HIP headers not found")
    exe = tmp_path / "host_tsan"
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=thread", "-fno-omit-frame-pointer",
                    "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
                    "-I", CSRC, "-o", str(exe), os.path.join(NATIVE, "host_sanitize.cpp"),
                    os.path.join(CSRC, "capi.cpp"), os.path.join(CSRC, "plan.cpp"), "-pthread"], check=True)
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1")
    res = subprocess.run([str(exe), "threads", "8", "48"], capture_output=True, text=True, timeout=600, env=env)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "ThreadSanitizer" not in out, out[-4000:]
    assert "0 launch contract problems, 0 failures" in out, out[-4000:]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc is not installed")
def test_oracle_under_sanitizers(tmp_path):
    exe = tmp_path / "oracle_sanitize"
    subprocess.run(["gcc", "-std=c11", *SAN, "-o", str(exe), os.path.join(NATIVE, "oracle_sanitize.c"),
                    os.path.join(ROOT, "oracle", "oracle.c"), "-lm"], check=True)
    rc, out = _run(exe)
    assert rc == 0, out[-4000:]
    assert "68 values of P, 0 failures" in out, out[-4000:]
