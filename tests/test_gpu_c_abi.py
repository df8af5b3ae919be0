"""The C ABI on the GPU from C: tests/native/c_abi_gpu.c (C99, gcc, linked
against libar.so and the HIP runtime; no Python or torch in the process)
allocates the rank buffers with hipMalloc, runs ar_execute /
ar_execute_batched on a stream of its own, and its results must equal the
oracle's bit for bit -- the Allreduce of Sec. 1 over the exchanges of
Sec. 5.3, through every kind of launch: step-wise with scratch, fused
bandwidth-optimal, the split pair at P = 127, latency-optimal batches,
rank slots on short blocks, and a plan whose k the cost model chose."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2004_09362_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2004_09362_amd")
SRC = os.path.join(ROOT, "tests", "native", "c_abi_gpu.c")

AUTO, STEPWISE, FUSED = 0, 1, 2

CASES = [
    # P, n, batch, stride, k, dtype, op, path, batched
    (7, 1000, 1, 1000, 5, "float32", "sum", STEPWISE, 0),
    (7, 1000, 1, 1000, 5, "float32", "sum", FUSED, 0),
    (3, 1024, 1, 1024, 2, "int32", "sum", AUTO, 0),
    (12, 106, 64, 106, 4, "float32", "sum", AUTO, 1),
    (24, 106, 33, 110, 10, "float32", "sum", AUTO, 1),
    (37, 4101, 1, 4101, -1, "int32", "max", AUTO, 0),
    (37, 4101, 3, 4200, -1, "float32", "sum", STEPWISE, 1),
    (127, 9219, 1, 9219, 14, "float32", "sum", AUTO, 0),
    (127, 9219, 1, 9219, 10, "float32", "sum", STEPWISE, 0),
    (127, 524295, 1, 524295, 14, "float32", "sum", AUTO, 0),  # 2 MiB per rank: split, destination-major copy
    (127, 524295, 1, 524295, 10, "float32", "sum", AUTO, 0),  # shifted at odd P: the rank-slot kernel
]


@pytest.fixture(scope="module")
def exe(tmp_path_factory):
    lib = os.path.join(LIBDIR, "libar.so")
    if not os.path.exists(lib):
        pytest.fail("libar.so is not built")
    out = tmp_path_factory.mktemp("cabi") / "c_abi_gpu"
    cmd = ["gcc", "-std=c99", "-O1", "-Wall", "-Wextra", "-Werror=implicit-function-declaration",
           "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROOT, "include"), "-I/opt/rocm/include", SRC,
           "-L" + LIBDIR, "-l:libar.so", "-Wl,-rpath," + LIBDIR, "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath,/opt/rocm/lib", "-o", str(out)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-3000:]
    return str(out)


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES, ids=lambda c: "P%d_n%d_b%d_k%d_%s_%s_path%d" % (c[0], c[1], c[2], c[4], c[5], c[6], c[7]))
def test_c_program_on_the_gpu(exe, tmp_path, case):
    P, n, batch, stride, k, dtype, op, path, batched = case
    extent = (batch - 1) * stride + n
    dt = np.dtype(dtype)
    dist = synth.Dist("randint", -1000, 1000) if dtype == "int32" else synth.Dist("normal", 0.0, 1.0)
    x = synth.host_ranks(synth.BASE_SEED + 77 + P, P, extent, dt, dist)
    inp, outp = tmp_path / "in.bin", tmp_path / "out.bin"
    hdr = np.array([P, n, batch, stride, k, 0 if dtype == "int32" else 1, 0 if op == "sum" else 1, path, batched],
                   dtype=np.int64)
    with open(inp, "wb") as fh:
        fh.write(hdr.tobytes())
        fh.write(np.ascontiguousarray(x).tobytes())
    print("c_abi_gpu case", case, flush=True)
    run = subprocess.run([exe, str(inp), str(outp)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    raw = np.fromfile(outp, dtype=np.uint8)
    got_k, got_path = np.frombuffer(raw[:16].tobytes(), dtype=np.int64)
    got = np.frombuffer(raw[16:].tobytes(), dtype=dt).reshape(P, extent)
    L = max(0, (P - 1).bit_length())
    if k >= 0:
        assert got_k == k
    else:
        assert L <= got_k <= 2 * L
    assert got_path == (path if path != AUTO else FUSED)
    # the oracle at the plan's k, instance by instance; gaps between instances untouched
    xi = np.stack([x[:, j * stride:j * stride + n] for j in range(batch)], axis=1)
    want = oracle.allreduce_batched(np.ascontiguousarray(xi), int(got_k), op)
    for j in range(batch):
        assert np.array_equal(got[:, j * stride:j * stride + n].view(np.uint32), want[:, j].view(np.uint32)), j
        if j + 1 < batch:
            gap = slice(j * stride + n, (j + 1) * stride)
            assert np.array_equal(got[:, gap].view(np.uint32), x[:, gap].view(np.uint32))
