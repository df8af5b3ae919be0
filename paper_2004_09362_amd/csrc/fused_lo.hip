// fused_lo.hip -- the fused latency-optimal kernel for small P.
//
// Kolmakov & Zhang, "A Generalization of the Allreduce Operation"
// (arXiv:2004.09362), Sec. 9.  fused_lo_kernel runs the whole
// latency-optimal schedule for one column of P values held in registers:
// the primed vector R[x] and the starred S[x] of every rank, updated as the
// reduction steps prescribe, then S[x] written to rank x.  The pairs
// combined are exactly those of the step-by-step path, so the results are
// bit-identical, but each input is read once and each output written once
// (2*P*n elements).  The latency-optimal tree of rank x is the same for
// every block, so many small instances form one flat column space with no
// block index: the kernel for many independent small messages (Sec. 1's
// 425-byte average).
//
// Compiled with packed-fp32 instructions disabled; only adds and compares.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "ar_internal.hpp"
#include "device_common.hpp"

namespace ar {

namespace {

constexpr int lo_L(int P) {
  int L = 0;
  while ((1 << L) < P) ++L;
  return L;
}
constexpr int lo_N(int P, int i) {
  int N = P;
  for (int j = 0; j < i; ++j) N -= N / 2;
  return N;
}

template <typename V, int OP>
struct Comb;
template <int OP>
struct Comb<float, OP> {
  __device__ __forceinline__ static float f(float a, float b) { return comb<OP>(a, b); }
};
template <int OP>
struct Comb<int32_t, OP> {
  __device__ __forceinline__ static int32_t f(int32_t a, int32_t b) { return comb<OP>(a, b); }
};

// Reduction step I of the latency-optimal schedule on one column: with
// f = floor(N_I/2), every rank receives the primed vector of rank x + f;
// starred sums take it on even N_I, primed sums on every step but the last.
// Before the first odd step S and R hold the same values, and the compiler
// computes their identical combinations once.
template <int P, int I, int OP, typename V>
__device__ __forceinline__ void lo_steps(V (&R)[P], V (&S)[P]) {
  constexpr int L = lo_L(P);
  if constexpr (I < L) {
    constexpr int N = lo_N(P, I);
    constexpr int f = N / 2;
    constexpr bool even = (N % 2) == 0;
    constexpr bool last = (I == L - 1);
    V Rn[P];
#pragma unroll
    for (int x = 0; x < P; ++x) {
      const V recv = R[(x + f) % P];
      if constexpr (even) S[x] = Comb<V, OP>::f(S[x], recv);
      if constexpr (!last) Rn[x] = Comb<V, OP>::f(R[x], recv);
    }
    if constexpr (!last) {
#pragma unroll
      for (int x = 0; x < P; ++x) R[x] = Rn[x];
    }
    lo_steps<P, I + 1, OP, V>(R, S);
  }
}

// MODE 1: contiguous instances, column g = element g (4-byte accesses; 16-byte
//         column groups measured 5-9% slower and are not built);
// MODE 2: any instance stride, column g = element g % n of instance g / n.
template <int P, typename T, int OP, int MODE, bool NT>
__global__ __launch_bounds__(kBlock) void fused_lo_kernel(const FusedArgs a) {
  const int64_t nthreads = int64_t(gridDim.x) * kBlock;
  for (int64_t g = int64_t(blockIdx.x) * kBlock + threadIdx.x; g < a.groups; g += nthreads) {
    int64_t e = g;
    if constexpr (MODE == 2) {
      const int64_t inst = g / a.n;
      e = inst * a.stride + (g - inst * a.n);
    }
    T R[P], S[P];
#pragma unroll
    for (int x = 0; x < P; ++x) {
      R[x] = ld1<NT>(reinterpret_cast<const T*>(a.user[x]) + e);
      S[x] = R[x];
    }
    lo_steps<P, 0, OP, T>(R, S);
#pragma unroll
    for (int x = 0; x < P; ++x) st1<NT>(reinterpret_cast<T*>(a.user[x]) + e, S[x]);
  }
}

template <int P, typename T, int OP>
int launch_fused_p(const FusedArgs& a, int mode, bool nt, int grid, hipStream_t s) {
  const dim3 g(grid), blk(kBlock);
  if (mode == 1) {
    if (nt) hipLaunchKernelGGL((fused_lo_kernel<P, T, OP, 1, true>), g, blk, a.lds, s, a);
    else hipLaunchKernelGGL((fused_lo_kernel<P, T, OP, 1, false>), g, blk, a.lds, s, a);
  } else if (mode == 2) {
    hipLaunchKernelGGL((fused_lo_kernel<P, T, OP, 2, false>), g, blk, a.lds, s, a);
  } else {
    return int(hipErrorInvalidValue);
  }
  return int(hipGetLastError());
}

template <typename T, int OP>
int launch_fused_t(const FusedArgs& a, int P, int mode, bool nt, int grid, hipStream_t s) {
  switch (P) {
#define AR_LO_CASE(PP) \
  case PP: return launch_fused_p<PP, T, OP>(a, mode, nt, grid, s);
    AR_LO_CASE(2) AR_LO_CASE(3) AR_LO_CASE(4) AR_LO_CASE(5) AR_LO_CASE(6) AR_LO_CASE(7) AR_LO_CASE(8)
    AR_LO_CASE(9) AR_LO_CASE(10) AR_LO_CASE(11) AR_LO_CASE(12) AR_LO_CASE(13) AR_LO_CASE(14)
    AR_LO_CASE(15) AR_LO_CASE(16)
#undef AR_LO_CASE
    default: return int(hipErrorInvalidValue);
  }
}

}  // namespace

int launch_fused_lo(const FusedArgs& a, int P, int dtype, int op, int mode, bool nt, int grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (dtype == 0)
    return op == 0 ? launch_fused_t<int32_t, 0>(a, P, mode, nt, grid, s) : launch_fused_t<int32_t, 1>(a, P, mode, nt, grid, s);
  return op == 0 ? launch_fused_t<float, 0>(a, P, mode, nt, grid, s) : launch_fused_t<float, 1>(a, P, mode, nt, grid, s);
}

}  // namespace ar
