// fused_bo.hpp -- column-fused bandwidth-optimal Allreduce kernel.
//
// Kolmakov & Zhang, "A Generalization of the Allreduce Operation"
// (arXiv:2004.09362), Sec. 7.  For block b, placement p of the reduction
// lives on rank b + p, so one element column of block b is the array
// W[p] = V_{b+p}[e], p = 0..P-1.  Reduction step i (N_i vectors, f_i =
// floor(N_i/2), c_i = ceil(N_i/2)) combines the kept placements
// [c_i - f_i, c_i) with the received [c_i, N_i): W[p] = W[p] (+) W[p + f_i].
// After ceil(log2 P) steps W[0] holds the reduction of the column, and the
// distribution phase hands that same value to every rank.  Doing this per
// column in registers combines exactly the operand pairs of the step-by-step
// schedule, in the same order, so the bits are identical -- but every input
// is read once and every output written once (2 * P * n elements of HBM
// traffic instead of 5 * (P - 1) * n).
//
// One wave covers 64 consecutive columns of one block of one instance, one
// 4-byte element per lane: the block, hence the rotation of the rank
// pointers, is uniform across the wave and every access is a coalesced
// 256-byte row of one rank buffer.  Blocks start at arbitrary elements, so
// the tiles of a block are laid on 256-byte boundaries of the buffer (the
// first and last tile of a block are partial): rows that straddled cache
// lines cost a third more line transfers, and much more when streamed
// nontemporally.  P is a template parameter so that W stays in registers
// with static indices.
#pragma once

#include "device_common.hpp"

namespace ar {

template <int N, int OP, typename T, int P>
__device__ __forceinline__ void bo_fold(T (&w)[P]) {
  if constexpr (N > 1) {
    constexpr int f = N / 2;
    constexpr int c = N - f;
#pragma unroll
    for (int j = c - f; j < c; ++j) w[j] = comb<OP>(w[j], w[j + f]);
    bo_fold<c, OP, T, P>(w);
  }
}

template <int P, typename T, int OP, bool NT>
__global__ __launch_bounds__(kBlock) void fused_bo_kernel(const ColArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t wave_in_block = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  for (uint32_t t = blockIdx.x * uint32_t(kWavesPerBlock) + wave_in_block; t < a.total_tiles;
       t += gridDim.x * uint32_t(kWavesPerBlock)) {
    const uint32_t seg = fdiv(t, a.tiles);  // seg = instance * P + block
    const uint32_t tile = t - seg * a.tiles.d;
    const uint32_t inst = fdiv(seg, a.pdiv);
    const int32_t b = int32_t(seg - inst * a.pdiv.d);
    const int64_t len = a.q + (b < a.m ? 1 : 0);
    const int64_t e0 = int64_t(inst) * a.stride + int64_t(b) * a.q + (b < a.m ? b : a.m);
    void* const* rot = a.user + b;  // rot[d] is rank (b + d) mod P
    // columns before the first 256-byte boundary of the root rank's row
    const int64_t lo = ((reinterpret_cast<uintptr_t>(rot[0]) >> 2) + e0) & (kWave - 1);
    const int64_t c = int64_t(tile) * kWave - lo + lane;
    if (c >= 0 && c < len) {
      const int64_t e = e0 + c;
      T w[P];
#pragma unroll
      for (int d = 0; d < P; ++d) w[d] = ld1<NT>(static_cast<const T*>(rot[d]) + e);
      bo_fold<P, OP, T, P>(w);
#pragma unroll
      for (int d = 0; d < P; ++d) st1<NT>(static_cast<T*>(rot[d]) + e, w[0]);
    }
  }
}

template <int P>
int launch_fused_bo(const ColArgs& a, int dtype, int op, bool nt, int grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const dim3 g(grid), blk(kBlock);
  if (dtype == 0) {
    if (op == 0) {
      if (nt) hipLaunchKernelGGL((fused_bo_kernel<P, int32_t, 0, true>), g, blk, 0, s, a);
      else hipLaunchKernelGGL((fused_bo_kernel<P, int32_t, 0, false>), g, blk, 0, s, a);
    } else {
      if (nt) hipLaunchKernelGGL((fused_bo_kernel<P, int32_t, 1, true>), g, blk, 0, s, a);
      else hipLaunchKernelGGL((fused_bo_kernel<P, int32_t, 1, false>), g, blk, 0, s, a);
    }
  } else {
    if (op == 0) {
      if (nt) hipLaunchKernelGGL((fused_bo_kernel<P, float, 0, true>), g, blk, 0, s, a);
      else hipLaunchKernelGGL((fused_bo_kernel<P, float, 0, false>), g, blk, 0, s, a);
    } else {
      if (nt) hipLaunchKernelGGL((fused_bo_kernel<P, float, 1, true>), g, blk, 0, s, a);
      else hipLaunchKernelGGL((fused_bo_kernel<P, float, 1, false>), g, blk, 0, s, a);
    }
  }
  return int(hipGetLastError());
}

}  // namespace ar
