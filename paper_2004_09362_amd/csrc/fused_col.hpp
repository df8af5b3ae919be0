// fused_col.hpp -- column-fused Allreduce kernels: every step of the
// schedule applied to element columns held in registers.
//
// fused_bo_kernel: bandwidth-optimal schedules (r = 0).
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
// With a.split set, only the root rank b receives the result and a second
// launch (broadcast.hip) copies it to the other ranks: the same bits, one
// more read and write of a block per column, but the reading and the writing
// of the P streams no longer interleave (see the broadcast kernel).
//
// One wave covers 64 consecutive columns of one block of one instance, one
// 4-byte element per lane: the block, hence the rotation of the rank
// pointers, is uniform across the wave and every access is a coalesced
// 256-byte row of one rank buffer.  Blocks start at arbitrary elements, so
// the tiles of a block are laid on 256-byte boundaries of the buffer (the
// first and last tile of a block are partial): rows that straddled cache
// lines cost a third more line transfers, and much more when streamed
// nontemporally.  Blocks of at most 64 elements (many small instances) are
// packed instead: a wave takes the same block of several instances, so the
// rotation stays uniform while the lanes fill (col_tile_column in
// device_common.hpp).  P is a template parameter so that W stays in
// registers with static indices.
#pragma once

#include <type_traits>
#include <utility>

#include "device_common.hpp"

namespace ar {

constexpr int col_L(int P) {
  int L = 0;
  while ((1 << L) < P) ++L;
  return L;
}

constexpr int col_N(int P, int i) {
  int N = P;
  for (int j = 0; j < i; ++j) N -= N / 2;
  return N;
}

// Placement whose starred result reaches placement q through the
// distribution phase, for 2^r shifted schedules (Secs. 7-8): placements
// [0, w) are held after the reduction; the reversed step i (run only when
// N_i exceeds the placements held so far, h) delivers [max(c_i, h), N_i)
// from placement q - f_i of rank x - f_i, i.e. from the same block.
constexpr int col_src(int P, int r, int q) {
  const int L = col_L(P);
  const int w = (1 << r) < P ? (1 << r) : P;
  int lo[16] = {}, hi[16] = {}, fs[16] = {};
  int k = 0, h = w;
  for (int i = L - 1; i >= 0; --i) {
    const int N = col_N(P, i);
    if (N <= h) continue;
    const int f = N / 2, c = N - f;
    lo[k] = c > h ? c : h;
    hi[k] = N;
    fs[k] = f;
    ++k;
    h = N;
  }
  for (int t = k - 1; t >= 0; --t)
    if (q >= lo[t] && q < hi[t]) q -= fs[t];
  return q;
}

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
    int32_t b;
    int64_t e;
    const bool live = col_tile_column(a, t, lane, b, e);
    void* const* rot = a.user + b;  // rot[d] is rank (b + d) mod P
    if (live) {
      T w[P];
#pragma unroll
      for (int d = 0; d < P; ++d) w[d] = ld1<NT>(static_cast<const T*>(rot[d]) + e);
      bo_fold<P, OP, T, P>(w);
      if (a.split) {
        st1<NT>(static_cast<T*>(rot[0]) + e, w[0]);
      } else {
#pragma unroll
        for (int d = 0; d < P; ++d) st1<NT>(static_cast<T*>(rot[d]) + e, w[0]);
      }
    }
  }
}

// With a.flat (latency-optimal plans) the tile loop runs over the flat
// columns of all instances with b = 0: rank q then stores S[q], the tree
// rooted at itself, which is the same for every block.  Many small
// instances (blocks of a few elements, or none) then fill whole waves.
//
// fused_mid_kernel: shifted (intermediate) and latency-optimal schedules,
// 1 <= r <= ceil(log2 P).  For block b the column is V[d] = V_{b+d}[e].  The
// primed sums R[d] and starred sums S[d] of every offset d follow the
// reduction steps of Secs. 8-9: with f = floor(N_i/2), S[d] takes R[d + f]
// when N_i is even and R[d] takes R[d + f] on every step but the last.
// S[s] is then the starred result of shift s, rooted at rank b + s -- the
// recursion does not depend on how many shifts are kept -- and rank b + q
// receives S[col_src(q)], the result the distribution phase brings it.
// All P starred sums are computed whatever r is (at most P(2L - 2)
// combines per column, far below the memory time), so one kernel per P
// serves every r, and the store pattern is picked by a uniform branch.
template <int P, int I, int OP, typename T>
__device__ __forceinline__ void mid_steps(T (&R)[P], T (&S)[P]) {
  constexpr int L = col_L(P);
  if constexpr (I < L) {
    constexpr int N = col_N(P, I);
    constexpr int f = N / 2;
    constexpr bool even = (N % 2) == 0;
    constexpr bool last = (I == L - 1);
    T Rn[P];
#pragma unroll
    for (int d = 0; d < P; ++d) {
      const T recv = R[(d + f) % P];
      if constexpr (even) S[d] = comb<OP>(S[d], recv);
      if constexpr (!last) Rn[d] = comb<OP>(R[d], recv);
    }
    if constexpr (!last) {
#pragma unroll
      for (int d = 0; d < P; ++d) R[d] = Rn[d];
    }
    mid_steps<P, I + 1, OP, T>(R, S);
  }
}

// Rank offset q stores S[col_src(q)]; the index is forced to a compile-time
// constant so the table never reaches memory.
template <int P, int RR, bool NT, typename T, int... Qs>
__device__ __forceinline__ void mid_store_seq(void* const* rot, int64_t e, const T (&S)[P],
                                              std::integer_sequence<int, Qs...>) {
  (st1<NT>(static_cast<T*>(rot[Qs]) + e, S[std::integral_constant<int, col_src(P, RR, Qs)>::value]), ...);
}

template <int P, int RR, bool NT, typename T>
__device__ __forceinline__ void mid_store(void* const* rot, int64_t e, const T (&S)[P]) {
  mid_store_seq<P, RR, NT, T>(rot, e, S, std::make_integer_sequence<int, P>{});
}

template <int P, int RR, bool NT, typename T>
__device__ __forceinline__ void mid_store_r(int r, void* const* rot, int64_t e, const T (&S)[P]) {
  if constexpr (RR <= col_L(P)) {
    if (r == RR) mid_store<P, RR, NT, T>(rot, e, S);
    else mid_store_r<P, RR + 1, NT, T>(r, rot, e, S);
  }
}

template <int P, typename T, int OP, bool NT>
__global__ __launch_bounds__(kBlock) void fused_mid_kernel(const ColArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t wave_in_block = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  for (uint32_t t = blockIdx.x * uint32_t(kWavesPerBlock) + wave_in_block; t < a.total_tiles;
       t += gridDim.x * uint32_t(kWavesPerBlock)) {
    int32_t b;
    int64_t e;
    bool live;
    if (a.flat) {  // r = L: flat columns, every rank's tree rooted at itself (b = 0)
      const uint32_t g = t * uint32_t(kWave) + uint32_t(lane);
      const uint32_t inst = fdiv(g, a.ndiv);
      b = 0;
      e = int64_t(inst) * a.stride + int64_t(g - inst * a.ndiv.d);
      live = g < a.flat_cols;
    } else {
      live = col_tile_column(a, t, lane, b, e);
    }
    void* const* rot = a.user + b;
    if (live) {
      T R[P], S[P];
#pragma unroll
      for (int d = 0; d < P; ++d) {
        R[d] = ld1<NT>(static_cast<const T*>(rot[d]) + e);
        S[d] = R[d];
      }
      mid_steps<P, 0, OP, T>(R, S);
      mid_store_r<P, 1, NT, T>(a.r, rot, e, S);
    }
  }
}

// fused_rot_kernel: batches of short blocks in rank slots over flat
// columns, for the cyclic butterfly plans with r < L (the bandwidth-optimal
// fold and the shifted recursion above) and the Ring; sums, and max where
// every rank receives one result.  Lane g holds element i of instance
// g / n; its block b follows from i.  It loads X[y] = V_y[e] for every rank
// y -- each load a whole 256-byte row of one rank buffer, whatever the
// blocks -- and rotates the column by b, X[p] <- X[b + p], so that X[p] is
// placement p's value, V_{b+p}, exactly as the block-tiled kernels read it
// through rotated pointers.  The fold, the recursion or the chain then
// combines the same operand pairs in the same order (the same bits, also
// for a max of signed zeros or NaNs).  The bandwidth-optimal and Ring
// result goes to every rank (with a.split, to rank 0 alone, and the
// broadcast copies it); in the shifted plan rank b + q receives
// S[col_src(q)], so the column of results is rotated back by b and rank y
// stores slot y.  A rotation by a per-lane amount is a
// log-depth network of static rotations by 2^j, each applied on the lanes
// whose amount has bit j set (P selects per stage; a stage no lane needs is
// skipped).

// Lanes whose bit in m is set take b, the others a: one v_cndmask_b32.  The
// instruction is written out because the compiler otherwise turned the
// selects of a rotation network into selects of array indices and rebuilt
// the network as duplicated select trees behind divergent branches (2761
// selects instead of 120 at P = 24, six times slower).
template <typename T>
__device__ __forceinline__ T lane_select(uint64_t m, T a, T b) {
  static_assert(sizeof(T) == 4, "4-byte elements");
  uint32_t r;
  asm("v_cndmask_b32 %0, %1, %2, %3"
      : "=v"(r)
      : "v"(__builtin_bit_cast(uint32_t, a)), "v"(__builtin_bit_cast(uint32_t, b)), "s"(m));
  return __builtin_bit_cast(T, r);
}

// X[p] <- X[(p + s) mod P] for the lane's s in [0, P).
template <int P, int K, typename T>
__device__ __forceinline__ void rotate_lanes(T (&X)[P], uint32_t s) {
  if constexpr ((1 << K) < P) {
    constexpr int sh = 1 << K;
    const uint64_t m = __builtin_amdgcn_ballot_w64(((s >> K) & 1u) != 0);
    if (m != 0) {
      T Y[P];
#pragma unroll
      for (int p = 0; p < P; ++p) Y[p] = lane_select(m, X[p], X[(p + sh) % P]);
#pragma unroll
      for (int p = 0; p < P; ++p) X[p] = Y[p];
    }
    rotate_lanes<P, K + 1, T>(X, s);
  }
}

// Shifted plan with RR removed distribution steps: slot q takes
// S[col_src(q)], the result that reaches placement q (compile-time indices).
template <int P, int RR, typename T, int... Qs>
__device__ __forceinline__ void rot_gather(T (&Z)[P], const T (&S)[P], std::integer_sequence<int, Qs...>) {
  ((Z[Qs] = S[std::integral_constant<int, col_src(P, RR, Qs)>::value]), ...);
}

// RR = 0: the bandwidth-optimal fold; RR >= 1: the shifted recursion with
// RR distribution steps removed; RR = -1: the Ring of Sec. 6, whose column
// is the chain acc = V_{b+d} (+) acc, d = 1 .. P-1, from V_b (the order of
// fused_ring_kernel), its result going to every rank.  RR is a template
// parameter so that the compiler drops the starred sums that no rank
// receives (all but 2^RR of them) and the primed sums that only feed those
// (at P = 127, RR = 4: 306 of 1524 combinations); with all of them kept,
// the P = 127 kernels spilled registers.  Loads and stores are always
// nontemporal: these launches stream short blocks of many instances once.
template <int P, int RR, typename T, int OP>
__global__ __launch_bounds__(kBlock) void fused_rot_kernel(const ColArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t wave_in_block = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  for (uint32_t t = blockIdx.x * uint32_t(kWavesPerBlock) + wave_in_block; t < a.total_tiles;
       t += gridDim.x * uint32_t(kWavesPerBlock)) {
    const uint32_t g = t * uint32_t(kWave) + uint32_t(lane);
    // tbl is a.user (t < 2^31); indexing it by t >> 31 keeps the compiler
    // from hoisting the P rank pointers out of the loop, where they would stay
    // live across iterations in SGPRs spilled to VGPR lanes
    void* const* tbl = a.user + (t >> 31);
    if (g < a.flat_cols) {
      const uint32_t inst = fdiv(g, a.ndiv);
      const uint32_t i = g - inst * a.ndiv.d;
      const uint32_t longer = uint32_t(a.m) * (uint32_t(a.q) + 1);  // elements in the blocks of q + 1
      const uint32_t b = i < longer ? fdiv(i, a.q1div) : uint32_t(a.m) + fdiv(i - longer, a.qdiv);
      const int64_t e = int64_t(inst) * a.stride + i;
      T X[P];
#pragma unroll
      for (int y = 0; y < P; ++y) X[y] = ld1<true>(static_cast<const T*>(tbl[y]) + e);
      rotate_lanes<P, 0, T>(X, b);
      if constexpr (RR <= 0) {
        T acc;
        if constexpr (RR < 0) {
          acc = X[0];
#pragma unroll
          for (int d = 1; d < P; ++d) acc = comb<OP>(X[d], acc);
        } else {
          bo_fold<P, OP, T, P>(X);
          acc = X[0];
        }
        if (a.split) {  // every rank receives acc: rank 0 holds it first, the broadcast copies it
          st1<true>(static_cast<T*>(tbl[0]) + e, acc);
        } else {
#pragma unroll
          for (int y = 0; y < P; ++y) st1<true>(static_cast<T*>(tbl[y]) + e, acc);
        }
      } else {
        T S[P];
#pragma unroll
        for (int d = 0; d < P; ++d) S[d] = X[d];
        mid_steps<P, 0, OP, T>(X, S);
        // rank b + q receives slot q: rotate the slots back by b, rank y stores slot y
        rot_gather<P, RR, T>(X, S, std::make_integer_sequence<int, P>{});
        rotate_lanes<P, 0, T>(X, b == 0 ? 0u : uint32_t(P) - b);
#pragma unroll
        for (int y = 0; y < P; ++y) st1<true>(static_cast<T*>(tbl[y]) + e, X[y]);
      }
    }
  }
}

template <int P, int RR, typename T, int OP>
int launch_rot_rr(const ColArgs& a, int grid, hipStream_t s) {
  if constexpr (RR < col_L(P)) {
    if (a.r == RR) {
      hipLaunchKernelGGL((fused_rot_kernel<P, RR, T, OP>), dim3(grid), dim3(kBlock), a.lds, s, a);
      return int(hipGetLastError());
    }
    return launch_rot_rr<P, RR + 1, T, OP>(a, grid, s);
  } else {
    return int(hipErrorInvalidValue);
  }
}

// Sums at every r; max (op 1) for the bandwidth-optimal fold and the Ring,
// whose ranks all receive one result, and at every r for P in
// [kRotMaxShiftedMinP, kRotMaxShiftedMaxP].  Elsewhere shifted max plans
// keep the block or packed tiles, which saves most of the max
// instantiations.
template <int P>
int launch_fused_rot(const ColArgs& a, int dtype, int op, bool ring, int grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const dim3 g(grid), blk(kBlock);
  if (op == 1) {
    if (ring) {
      if (dtype == 0) hipLaunchKernelGGL((fused_rot_kernel<P, -1, int32_t, 1>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_rot_kernel<P, -1, float, 1>), g, blk, a.lds, s, a);
    } else if constexpr (P >= kRotMaxShiftedMinP && P <= kRotMaxShiftedMaxP) {
      return dtype == 0 ? launch_rot_rr<P, 0, int32_t, 1>(a, grid, s) : launch_rot_rr<P, 0, float, 1>(a, grid, s);
    } else {
      if (a.r != 0) return int(hipErrorInvalidValue);
      if (dtype == 0) hipLaunchKernelGGL((fused_rot_kernel<P, 0, int32_t, 1>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_rot_kernel<P, 0, float, 1>), g, blk, a.lds, s, a);
    }
    return int(hipGetLastError());
  }
  if (op != 0) return int(hipErrorInvalidValue);
  if (ring) {
    if (dtype == 0) hipLaunchKernelGGL((fused_rot_kernel<P, -1, int32_t, 0>), g, blk, a.lds, s, a);
    else hipLaunchKernelGGL((fused_rot_kernel<P, -1, float, 0>), g, blk, a.lds, s, a);
    return int(hipGetLastError());
  }
  return dtype == 0 ? launch_rot_rr<P, 0, int32_t, 0>(a, grid, s) : launch_rot_rr<P, 0, float, 0>(a, grid, s);
}

template <int P>
int launch_fused_bo(const ColArgs& a, int dtype, int op, bool nt, int grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const dim3 g(grid), blk(kBlock);
  if (dtype == 0) {
    if (op == 0) {
      if (nt) hipLaunchKernelGGL((fused_bo_kernel<P, int32_t, 0, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_bo_kernel<P, int32_t, 0, false>), g, blk, a.lds, s, a);
    } else {
      if (nt) hipLaunchKernelGGL((fused_bo_kernel<P, int32_t, 1, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_bo_kernel<P, int32_t, 1, false>), g, blk, a.lds, s, a);
    }
  } else {
    if (op == 0) {
      if (nt) hipLaunchKernelGGL((fused_bo_kernel<P, float, 0, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_bo_kernel<P, float, 0, false>), g, blk, a.lds, s, a);
    } else {
      if (nt) hipLaunchKernelGGL((fused_bo_kernel<P, float, 1, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_bo_kernel<P, float, 1, false>), g, blk, a.lds, s, a);
    }
  }
  return int(hipGetLastError());
}

}  // namespace ar

namespace ar {

template <int P>
int launch_fused_mid(const ColArgs& a, int dtype, int op, bool nt, int grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const dim3 g(grid), blk(kBlock);
  if (dtype == 0) {
    if (op == 0) {
      if (nt) hipLaunchKernelGGL((fused_mid_kernel<P, int32_t, 0, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_mid_kernel<P, int32_t, 0, false>), g, blk, a.lds, s, a);
    } else {
      if (nt) hipLaunchKernelGGL((fused_mid_kernel<P, int32_t, 1, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_mid_kernel<P, int32_t, 1, false>), g, blk, a.lds, s, a);
    }
  } else {
    if (op == 0) {
      if (nt) hipLaunchKernelGGL((fused_mid_kernel<P, float, 0, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_mid_kernel<P, float, 0, false>), g, blk, a.lds, s, a);
    } else {
      if (nt) hipLaunchKernelGGL((fused_mid_kernel<P, float, 1, true>), g, blk, a.lds, s, a);
      else hipLaunchKernelGGL((fused_mid_kernel<P, float, 1, false>), g, blk, a.lds, s, a);
    }
  }
  return int(hipGetLastError());
}

}  // namespace ar
