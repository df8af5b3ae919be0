/* c_abi_gpu.c -- a C99 caller of libar.so on the GPU, with no Python and no
 * torch: it allocates every rank buffer itself (hipMalloc), runs one
 * Allreduce through ar_execute or ar_execute_batched on a stream it creates,
 * and writes the results back for the test to compare with the oracle.
 *
 * Usage: c_abi_gpu IN OUT
 *   IN:  int64 header {P, n, batch, stride, k, dtype, op, path, batched},
 *        then P rank extents of (batch - 1) * stride + n 4-byte elements.
 *        k = -1 asks for AR_K_AUTO; path is an ar_path; batched = 0 calls
 *        ar_execute (batch 1), 1 calls ar_execute_batched.
 *   OUT: int64 {k, exec_path} of the plan, then the P extents after the call.
 * Exit status 0 on success; 2 with ar_last_error_message() on a library
 * error; 3 on a HIP or file error. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "ar.h"

#define HIP_OK(call)                                                                 \
  do {                                                                               \
    hipError_t e_ = (call);                                                          \
    if (e_ != hipSuccess) {                                                          \
      fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));              \
      return 3;                                                                      \
    }                                                                                \
  } while (0)

#define AR_OK_OR_FAIL(call)                                                          \
  do {                                                                               \
    ar_status s_ = (call);                                                           \
    if (s_ != AR_OK) {                                                               \
      fprintf(stderr, "%s: %s (%s)\n", #call, ar_last_error_message(),             \
              ar_status_string(s_));                                                 \
      return 2;                                                                      \
    }                                                                                \
  } while (0)

int main(int argc, char** argv) {
  int64_t h[9];
  FILE* f;
  int32_t P, x;
  int64_t n, batch, stride, extent;
  uint32_t* host;
  void* bufs[128];
  ar_plan* plan = NULL;
  ar_stats st;
  hipStream_t stream;
  int64_t out_hdr[2];

  if (argc != 3) return 3;
  f = fopen(argv[1], "rb");
  if (!f || fread(h, sizeof h, 1, f) != 1) return 3;
  P = (int32_t)h[0];
  n = h[1];
  batch = h[2];
  stride = h[3];
  if (P < 1 || P > 128 || n < 1 || batch < 1 || stride < n) return 3;
  extent = (batch - 1) * stride + n;
  host = (uint32_t*)malloc((size_t)P * (size_t)extent * 4);
  if (!host || fread(host, 4, (size_t)P * (size_t)extent, f) != (size_t)P * (size_t)extent) return 3;
  fclose(f);

  for (x = 0; x < P; ++x) {
    HIP_OK(hipMalloc(&bufs[x], (size_t)extent * 4));
    HIP_OK(hipMemcpy(bufs[x], host + (size_t)x * (size_t)extent, (size_t)extent * 4, hipMemcpyHostToDevice));
  }
  HIP_OK(hipStreamCreate(&stream));

  AR_OK_OR_FAIL(ar_plan_create(P, n, (ar_dtype)h[5], (ar_op)h[6], (int32_t)h[4], &plan));
  if (h[7] != AR_PATH_AUTO) AR_OK_OR_FAIL(ar_plan_set_path(plan, (ar_path)h[7]));
  AR_OK_OR_FAIL(ar_plan_stats(plan, &st));
  if (h[8])
    AR_OK_OR_FAIL(ar_execute_batched(plan, bufs, batch, stride, stream));
  else
    AR_OK_OR_FAIL(ar_execute(plan, bufs, stream));
  HIP_OK(hipStreamSynchronize(stream));

  for (x = 0; x < P; ++x)
    HIP_OK(hipMemcpy(host + (size_t)x * (size_t)extent, bufs[x], (size_t)extent * 4, hipMemcpyDeviceToHost));
  out_hdr[0] = st.k;
  out_hdr[1] = st.exec_path;
  f = fopen(argv[2], "wb");
  if (!f || fwrite(out_hdr, sizeof out_hdr, 1, f) != 1 ||
      fwrite(host, 4, (size_t)P * (size_t)extent, f) != (size_t)P * (size_t)extent)
    return 3;
  fclose(f);

  ar_plan_destroy(plan);
  HIP_OK(hipStreamDestroy(stream));
  for (x = 0; x < P; ++x) HIP_OK(hipFree(bufs[x]));
  free(host);
  printf("ok P=%d n=%lld batch=%lld k=%d path=%d\n", P, (long long)n, (long long)batch, st.k, st.exec_path);
  return 0;
}
