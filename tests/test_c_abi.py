"""The C ABI used from C: a C99 program includes include/ar.h, links
libar.so directly (no Python, no torch) and exercises every entry point that
needs no device memory -- plan construction for each group and schedule,
the automatic step count, stats, launch introspection, the cost model, and
the argument errors that are reported before any launch.  No GPU is needed;
nothing is launched (tests/test_gpu_c_abi.py runs a C program on the GPU)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2004_09362_amd")

PROG = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
#include "ar.h"

static int fails = 0;
#define CHECK(c) do { if (!(c)) { printf("FAIL line %d: %s\n", __LINE__, #c); ++fails; } } while (0)

int main(void) {
  ar_plan* p = NULL;
  ar_stats st;
  int32_t nl = 0;

  /* cyclic butterfly, P = 7, k = 5 (one distribution step removed) */
  CHECK(ar_plan_create(7, 1000, AR_FLOAT32, AR_SUM, 5, &p) == AR_OK && p != NULL);
  CHECK(ar_plan_stats(p, &st) == AR_OK);
  CHECK(st.P == 7 && st.L == 3 && st.k == 5 && st.r == 1 && st.w == 2);
  CHECK(st.rs_steps == 3 && st.ag_steps == 2 && st.fused_ok == 1);
  CHECK(st.group == AR_GROUP_CYCLIC && st.schedule == AR_SCHEDULE_BUTTERFLY);
  CHECK(st.bytes_pulled_total == st.blocks_pulled_per_rank * st.n * 4);
  CHECK(ar_plan_num_launches(p, &nl) == AR_OK && nl == 5);
  {
    ar_launch_desc d;
    ar_range_desc r[8];
    CHECK(ar_plan_launch(p, 0, &d, r, 8) == AR_OK && d.phase == 0 && d.n_ranges >= 1);
    CHECK(ar_plan_launch(p, nl - 1, &d, r, 8) == AR_OK && d.phase == 1 && r[0].kind == AR_KIND_COPY);
    CHECK(ar_plan_launch(p, nl, &d, r, 8) == AR_ERR_INVALID_ARG);
  }
  CHECK(ar_plan_set_path(p, AR_PATH_STEPWISE) == AR_OK);
  CHECK(ar_plan_set_path(p, (ar_path)7) == AR_ERR_INVALID_ARG);
  {
    double t = 0;
    CHECK(ar_plan_model_time(p, 1e-6, 1e-9, 0.0, &t) == AR_OK && t > 5e-6);
  }
  /* argument errors reported before any launch */
  {
    void* tbl[7] = {(void*)0x10000, (void*)0x20000, NULL, (void*)0x40000, (void*)0x50000, (void*)0x60000,
                    (void*)0x70000};
    CHECK(ar_execute(p, tbl, NULL) == AR_ERR_INVALID_ARG);
    CHECK(strlen(ar_last_error()) > 0);
    tbl[2] = (void*)0x30002;
    CHECK(ar_execute(p, tbl, NULL) == AR_ERR_INVALID_ARG);
    tbl[2] = (void*)0x20100; /* overlaps rank 1's 4000 bytes */
    CHECK(ar_execute(p, tbl, NULL) == AR_ERR_ALIAS);
    CHECK(ar_execute(p, NULL, NULL) == AR_ERR_INVALID_ARG);
    CHECK(ar_execute_batched(p, tbl, 0, 1000, NULL) == AR_ERR_INVALID_ARG);
    CHECK(ar_execute_batched(p, tbl, 2, 999, NULL) == AR_ERR_INVALID_ARG);
  }
  ar_plan_destroy(p);

  /* n = 0: nothing is touched, the pointers may be NULL */
  CHECK(ar_plan_create(5, 0, AR_INT32, AR_MAX, 3, &p) == AR_OK);
  {
    void* tbl[5] = {NULL, NULL, NULL, NULL, NULL};
    CHECK(ar_execute(p, tbl, NULL) == AR_OK);
  }
  ar_plan_destroy(p);

  /* XOR group: Recursive Halving, hybrid and Recursive Doubling at P = 8 */
  {
    const int64_t want_blocks[4] = {24, 16, 14, 14}; /* k = 3, 4, 5, 6 */
    for (int32_t k = 3; k <= 6; ++k) {
      CHECK(ar_plan_create_ex(8, 800, AR_INT32, AR_SUM, k, AR_GROUP_XOR, AR_SCHEDULE_BUTTERFLY, &p) == AR_OK);
      CHECK(ar_plan_stats(p, &st) == AR_OK);
      CHECK(st.group == AR_GROUP_XOR && st.k == k && st.blocks_pulled_per_rank == want_blocks[k - 3]);
      ar_plan_destroy(p);
    }
  }
  /* Ring, P = 12: 2(P-1) single-block steps */
  CHECK(ar_plan_create_ex(12, 1200, AR_FLOAT32, AR_MAX, 22, AR_GROUP_CYCLIC, AR_SCHEDULE_RING, &p) == AR_OK);
  CHECK(ar_plan_stats(p, &st) == AR_OK);
  CHECK(st.schedule == AR_SCHEDULE_RING && st.launches == 22 && st.blocks_pulled_per_rank == 22);
  CHECK(st.combines_per_rank == 11 && st.workspace_bytes == 0 && st.hbm_bytes_stepwise == 5LL * 11 * 1200 * 4);
  ar_plan_destroy(p);

  /* rejected plans leave *out_plan NULL */
  p = (ar_plan*)0x1;
  CHECK(ar_plan_create_ex(12, 10, AR_FLOAT32, AR_SUM, 4, AR_GROUP_XOR, AR_SCHEDULE_BUTTERFLY, &p) == AR_ERR_INVALID_ARG);
  CHECK(p == NULL);
  CHECK(ar_plan_create_ex(8, 10, AR_FLOAT32, AR_SUM, 3, AR_GROUP_CYCLIC, AR_SCHEDULE_RING, &p) == AR_ERR_INVALID_ARG);
  CHECK(ar_plan_create(7, 10, (ar_dtype)5, AR_SUM, 3, &p) == AR_ERR_UNSUPPORTED);
  CHECK(ar_plan_create(7, 10, AR_FLOAT32, AR_SUM, 2, &p) == AR_ERR_INVALID_ARG);
  CHECK(ar_plan_create(7, 10, AR_FLOAT32, AR_SUM, 3, NULL) == AR_ERR_INVALID_ARG);
  CHECK(ar_plan_stats(NULL, &st) == AR_ERR_INVALID_ARG);
  ar_plan_destroy(NULL);

  /* cost model: Table 2 parameters, the 425-byte message picks k = L */
  {
    int32_t k = 0;
    double r = 0, t = 0;
    CHECK(ar_model_best_k(127, 425.0, 3e-5, 1e-8, 2e-10, &k, &r) == AR_OK && k == 7);
    CHECK(ar_model_time(127, 425.0, 14, 3e-5, 1e-8, 2e-10, &t) == AR_OK && t > 14 * 3e-5);
    CHECK(ar_model_time(127, 425.0, 15, 3e-5, 1e-8, 2e-10, &t) == AR_ERR_INVALID_ARG);
  }
  /* automatic step count and path: the sentinel and the explicit call */
  {
    ar_model_params mp;
    double ts = 0, tf = 0;
    CHECK(ar_model_default_params(&mp) == AR_OK && mp.step_alpha > 0 && mp.fused_bytes_per_s > 0);
    CHECK(ar_plan_create(37, 1 << 20, AR_FLOAT32, AR_SUM, AR_K_AUTO, &p) == AR_OK);
    CHECK(ar_plan_stats(p, &st) == AR_OK && st.k >= 6 && st.k <= 12 && st.exec_path == AR_PATH_FUSED);
    CHECK(st.hbm_bytes_algorithmic == st.hbm_bytes_stepwise);
    CHECK(ar_plan_model_seconds(p, &mp, 1, AR_PATH_STEPWISE, &ts) == AR_OK);
    CHECK(ar_plan_model_seconds(p, NULL, 1, AR_PATH_FUSED, &tf) == AR_OK && tf < ts);
    ar_plan_destroy(p);
    mp.fused_bytes_per_s = 1.0; /* a fused path this slow loses: the plan runs step by step */
    CHECK(ar_plan_create_auto(37, 1 << 20, AR_FLOAT32, AR_SUM, AR_GROUP_CYCLIC, 1, AR_PATH_AUTO, &mp, &p) == AR_OK);
    CHECK(ar_plan_stats(p, &st) == AR_OK && st.exec_path == AR_PATH_STEPWISE);
    ar_plan_destroy(p);
    mp.step_alpha = -1.0;
    CHECK(ar_plan_create_auto(37, 100, AR_FLOAT32, AR_SUM, AR_GROUP_CYCLIC, 1, AR_PATH_AUTO, &mp, &p) ==
          AR_ERR_INVALID_ARG);
    CHECK(strlen(ar_last_error_message()) > 0 && strcmp(ar_last_error_message(), ar_last_error()) == 0);
  }
  CHECK(strcmp(ar_status_string(AR_OK), "ok") == 0);
  CHECK(strcmp(ar_status_string((ar_status)42), "unknown status") == 0);
  printf("%d failures\n", fails);
  return fails != 0;
}
"""


def test_c_program_uses_the_abi(tmp_path):
    lib = os.path.join(LIBDIR, "libar.so")
    if not os.path.exists(lib):
        pytest.fail("libar.so is not built")
    src = tmp_path / "abi.c"
    src.write_text(PROG)
    exe = tmp_path / "abi"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror=implicit-function-declaration",
           "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROOT, "include"), "-I/opt/rocm/include", str(src),
           "-L" + LIBDIR, "-l:libar.so", "-Wl,-rpath," + LIBDIR, "-lm", "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-3000:]
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "0 failures" in run.stdout
