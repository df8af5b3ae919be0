// fused_group.hip -- column-fused kernels of the schedules the paper derives
// as special cases of its algorithm (Kolmakov & Zhang, "A Generalization of
// the Allreduce Operation", arXiv:2004.09362):
//
// fused_xor_kernel: the butterfly schedules over the group of Table 1b
// (power-of-two P, t_k(x) = x XOR k) -- Recursive Halving for k = 2L
// (Sec. 7, closing remark), Recursive Doubling for k = L (Sec. 9, closing
// remark) and the hybrid between them (Sec. 8).  Placement p of rank x holds
// block x XOR p and step i (f_i = P / 2^(i+1)) pulls from rank x XOR f_i.
// For block b the reduction of one element column, written by rank rather
// than by placement, is: while f >= w = 2^r, every pair of slots {y, y|f}
// (bit f of y clear) combines into slot y, the kept operand being the rank
// whose bit f agrees with b's (it holds the block's placement in [0, f));
// after these halving levels slot y < w holds the partial sum rooted at the
// rank of b's w-group whose low bits are y.  While f < w every slot y < w
// combines with slot y XOR f, own value first (the doubling levels).  Rank
// x's result is the one rooted at the rank of b's w-group with x's low
// bits: slot x mod w.  The pairs and operand order are exactly those of the
// step-by-step schedule, so the bits are identical.  Because the slots are
// ranks, every block uses the same pointer table and all indices are
// compile-time constants; only the operand order of a halving level depends
// on b, through a wave-uniform select.
//
// fused_ring_kernel: the Ring (Sec. 6).  For block b, reduction step i
// combines rank b+i+1's own value with the partial sum of ranks b..b+i
// received from rank b+i, so one column is the chain
// acc = V_{b+d} (+) acc, d = 1 .. P-1, starting from V_b, and the P - 1
// distribution steps hand acc to every rank.
//
// Both read every input once and write every output once (2 * P * n
// elements), one 4-byte element per lane, 64 consecutive columns of one
// block per wave, tiles laid on 256-byte boundaries of the block's root rank
// buffer, or one short block of several instances per wave -- the tiling of
// the cyclic column kernels (col_tile_column, device_common.hpp).  Where
// every rank receives the same result (the Ring, Recursive Halving) a split
// launch stores it to the root rank b only and broadcast.hip copies it on.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "ar_internal.hpp"
#include "device_common.hpp"

namespace ar {

namespace {

constexpr int xor_L(int P) {
  int L = 0;
  while ((1 << L) < P) ++L;
  return L;
}

// Halving levels f = F, F/2, ..., W: slot y (< f) keeps the pair {y, y|f}.
// The operand order is a wave-uniform branch, so each level updates its
// slots in place (a per-pair select had doubled the live registers).
template <int P, int W, int F, int OP, typename T>
__device__ __forceinline__ void xor_halving(T (&X)[P], uint32_t b) {
  if constexpr (F >= W && F >= 1) {
    if (b & uint32_t(F)) {  // the kept operand is slot y|f
#pragma unroll
      for (int y = 0; y < F; ++y) X[y] = comb<OP>(X[y + F], X[y]);
    } else {
#pragma unroll
      for (int y = 0; y < F; ++y) X[y] = comb<OP>(X[y], X[y + F]);
    }
    xor_halving<P, W, F / 2, OP, T>(X, b);
  }
}

// Doubling levels f = F, F/2, ..., 1 over the W held slots.
template <int P, int W, int F, int OP, typename T>
__device__ __forceinline__ void xor_doubling(T (&X)[P]) {
  if constexpr (F >= 1) {
#pragma unroll
    for (int y = 0; y < W; ++y) {
      if ((y & F) == 0) {
        const T u = X[y], v = X[y | F];
        X[y] = comb<OP>(u, v);
        X[y | F] = comb<OP>(v, u);
      }
    }
    xor_doubling<P, W, F / 2, OP, T>(X);
  }
}

template <int P, int R, typename T, int OP, bool NT>
__global__ __launch_bounds__(kBlock) void fused_xor_kernel(const ColArgs a) {
  constexpr int W = 1 << R;
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t wave_in_block = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  for (uint32_t t = blockIdx.x * uint32_t(kWavesPerBlock) + wave_in_block; t < a.total_tiles;
       t += gridDim.x * uint32_t(kWavesPerBlock)) {
    // The rank table is the same for every tile.  t < 2^31, so tbl is
    // a.user; indexing by t >> 31 keeps the compiler from hoisting the P
    // pointer loads out of the loop, which would keep them live across
    // iterations (spilling SGPRs into VGPRs and costing occupancy).
    void* const* tbl = a.user + (t >> 31);
    int32_t b;
    int64_t e;
    bool live;
    // Flat columns (batches of short blocks, and Recursive Doubling): the
    // block only orders the operands of a halving pair, which a sum does
    // not see, so sums and Recursive Doubling leave it out; a max takes the
    // lane's own block (the halving's order then differs from lane to lane).
    if (a.flat) {
      const uint32_t g = t * uint32_t(kWave) + uint32_t(lane);
      const uint32_t inst = fdiv(g, a.ndiv);
      const uint32_t i = g - inst * a.ndiv.d;
      b = 0;
      if constexpr (OP != 0 && R != xor_L(P)) {
        const uint32_t longer = uint32_t(a.m) * (uint32_t(a.q) + 1);  // elements in the blocks of q + 1
        b = int32_t(i < longer ? fdiv(i, a.q1div) : uint32_t(a.m) + fdiv(i - longer, a.qdiv));
      }
      e = int64_t(inst) * a.stride + int64_t(i);
      live = g < a.flat_cols;
    } else {
      live = col_tile_column(a, t, lane, b, e);
    }
    if (live) {
      T X[P];
#pragma unroll
      for (int y = 0; y < P; ++y) X[y] = ld1<NT>(static_cast<const T*>(tbl[y]) + e);
      xor_halving<P, W, P / 2, OP, T>(X, uint32_t(b));
      xor_doubling<P, W, W / 2, OP, T>(X);
      if (W == 1 && a.split) {  // Recursive Halving: one result, held first by rank b (rank 0 on flat columns)
        st1<NT>(static_cast<T*>(tbl[a.flat ? 0 : b]) + e, X[0]);
      } else {
#pragma unroll
        for (int x = 0; x < P; ++x) st1<NT>(static_cast<T*>(tbl[x]) + e, X[x & (W - 1)]);
      }
    }
  }
}

constexpr int kRingChunk = 16;

// NC chunks of 16 ranks: the kernel serves 16 (NC - 1) + 1 < P <= 16 NC + 1,
// so every load and store has a compile-time slot and a wave-uniform guard,
// and all P loads of a column are in flight before the chain starts.
template <int NC, typename T, int OP, bool NT>
__global__ __launch_bounds__(kBlock) void fused_ring_kernel(const ColArgs a) {
  constexpr int D = NC * kRingChunk;  // ranks after the root, upper bound
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t wave_in_block = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int32_t P = a.P;
  for (uint32_t t = blockIdx.x * uint32_t(kWavesPerBlock) + wave_in_block; t < a.total_tiles;
       t += gridDim.x * uint32_t(kWavesPerBlock)) {
    int32_t b;
    int64_t e;
    const bool live = col_tile_column(a, t, lane, b, e);
    void* const* rot = a.user + b;  // rot[d] is rank (b + d) mod P
    if (live) {
      T acc = ld1<NT>(static_cast<const T*>(rot[0]) + e);
      T v[D];
#pragma unroll
      for (int d = 1; d <= D; ++d)
        if (d < P) v[d - 1] = ld1<NT>(static_cast<const T*>(rot[d]) + e);
#pragma unroll
      for (int d = 1; d <= D; ++d)
        if (d < P) acc = comb<OP>(v[d - 1], acc);
      if (a.split) {
        st1<NT>(static_cast<T*>(rot[0]) + e, acc);
      } else {
#pragma unroll
        for (int d = 0; d <= D; ++d)
          if (d < P) st1<NT>(static_cast<T*>(rot[d]) + e, acc);
      }
    }
  }
}

template <int NC>
int launch_ring_nc(const ColArgs& a, int dtype, int op, bool nt, int grid, hipStream_t s) {
  const dim3 g(grid), blk(kBlock);
  if (dtype == 0) {
    if (op == 0) {
      if (nt) hipLaunchKernelGGL((fused_ring_kernel<NC, int32_t, 0, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_ring_kernel<NC, int32_t, 0, false>), g, blk, a.lds, s, a);
    } else {
      if (nt) hipLaunchKernelGGL((fused_ring_kernel<NC, int32_t, 1, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_ring_kernel<NC, int32_t, 1, false>), g, blk, a.lds, s, a);
    }
  } else {
    if (op == 0) {
      if (nt) hipLaunchKernelGGL((fused_ring_kernel<NC, float, 0, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_ring_kernel<NC, float, 0, false>), g, blk, a.lds, s, a);
    } else {
      if (nt) hipLaunchKernelGGL((fused_ring_kernel<NC, float, 1, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_ring_kernel<NC, float, 1, false>), g, blk, a.lds, s, a);
    }
  }
  return int(hipGetLastError());
}

template <int P, int R>
int launch_xor_pr(const ColArgs& a, int dtype, int op, bool nt, int grid, hipStream_t s) {
  const dim3 g(grid), blk(kBlock);
  if (dtype == 0) {
    if (op == 0) {
      if (nt) hipLaunchKernelGGL((fused_xor_kernel<P, R, int32_t, 0, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_xor_kernel<P, R, int32_t, 0, false>), g, blk, a.lds, s, a);
    } else {
      if (nt) hipLaunchKernelGGL((fused_xor_kernel<P, R, int32_t, 1, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_xor_kernel<P, R, int32_t, 1, false>), g, blk, a.lds, s, a);
    }
  } else {
    if (op == 0) {
      if (nt) hipLaunchKernelGGL((fused_xor_kernel<P, R, float, 0, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_xor_kernel<P, R, float, 0, false>), g, blk, a.lds, s, a);
    } else {
      if (nt) hipLaunchKernelGGL((fused_xor_kernel<P, R, float, 1, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_xor_kernel<P, R, float, 1, false>), g, blk, a.lds, s, a);
    }
  }
  return int(hipGetLastError());
}

template <int P, int R>
int launch_xor_r(const ColArgs& a, int dtype, int op, bool nt, int grid, hipStream_t s) {
  if constexpr ((1 << R) <= P) {
    if (a.r == R) return launch_xor_pr<P, R>(a, dtype, op, nt, grid, s);
    return launch_xor_r<P, R + 1>(a, dtype, op, nt, grid, s);
  } else {
    return int(hipErrorInvalidValue);
  }
}

}  // namespace

int launch_fused_xor(const ColArgs& a, int P, int dtype, int op, bool nt, int grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  switch (P) {
    case 2: return launch_xor_r<2, 0>(a, dtype, op, nt, grid, s);
    case 4: return launch_xor_r<4, 0>(a, dtype, op, nt, grid, s);
    case 8: return launch_xor_r<8, 0>(a, dtype, op, nt, grid, s);
    case 16: return launch_xor_r<16, 0>(a, dtype, op, nt, grid, s);
    case 32: return launch_xor_r<32, 0>(a, dtype, op, nt, grid, s);
    case 64: return launch_xor_r<64, 0>(a, dtype, op, nt, grid, s);
    case 128: return launch_xor_r<128, 0>(a, dtype, op, nt, grid, s);
    default: return int(hipErrorInvalidValue);
  }
}

int launch_fused_ring(const ColArgs& a, int dtype, int op, bool nt, int grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  switch ((a.P - 2) / kRingChunk) {  // P - 1 ranks after the root, in chunks of 16
    case 0: return launch_ring_nc<1>(a, dtype, op, nt, grid, s);
    case 1: return launch_ring_nc<2>(a, dtype, op, nt, grid, s);
    case 2: return launch_ring_nc<3>(a, dtype, op, nt, grid, s);
    case 3: return launch_ring_nc<4>(a, dtype, op, nt, grid, s);
    case 4: return launch_ring_nc<5>(a, dtype, op, nt, grid, s);
    case 5: return launch_ring_nc<6>(a, dtype, op, nt, grid, s);
    case 6: return launch_ring_nc<7>(a, dtype, op, nt, grid, s);
    case 7: return launch_ring_nc<8>(a, dtype, op, nt, grid, s);
    default: return int(hipErrorInvalidValue);
  }
}

}  // namespace ar
