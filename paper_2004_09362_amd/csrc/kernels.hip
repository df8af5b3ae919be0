// kernels.hip -- the step kernel of the generalized Allreduce for CDNA4
// (gfx950).
//
// Kolmakov & Zhang, "A Generalization of the Allreduce Operation"
// (arXiv:2004.09362).  step_kernel runs one communication step of the
// schedule (Secs. 6-9): every rank x, for each of its placements p in the
// launch's ranges, combines (or copies) block b = (x - p) mod P of its own
// buffer with the same block of rank (x + delta) mod P (in the XOR group:
// block x XOR p, rank x XOR delta).  The work is pure streaming -- three
// (copy: two, dual: five) block-sized HBM accesses per item, one add per
// element -- so the kernel is built for HBM bandwidth: 64-lane waves,
// 16-byte loads, several loads in flight per lane before the first store,
// and no LDS (every byte is used exactly once, there is nothing to share
// across lanes).  step_merged_kernel runs the same step for short blocks:
// each range's run of consecutive blocks of a rank as one flat space, so
// that batches of small instances fill their waves.
//
// The fused kernels are in fused_lo.hip (latency-optimal, small P, no block
// tiling), fused_col.hpp (column-fused, any P and k) and fused_group.hip
// (XOR group and Ring).
//
// Compiled with packed-fp32 instructions disabled; only adds and compares,
// so no contraction question arises.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "ar_internal.hpp"
#include "device_common.hpp"

namespace ar {

namespace {

template <typename T>
__device__ __forceinline__ T* buf_ptr(const StepArgs& a, int32_t buf, int32_t rank) {
  if (buf == kBufU) return reinterpret_cast<T*>(a.user[rank]);
  return reinterpret_cast<T*>(a.scratch[buf - 1]) + int64_t(rank) * a.scratch_rank_stride;
}

// One wave tile of one segment -- one block of one rank for one placement.
// The pointers are at the segment's first element; e0 is that element's
// index inside the rank buffer, which fixes its 16-byte phase (all buffers
// share it).  Vector path: the 16-byte aligned body is cut into 1 KB tiles
// that start on 128-byte lines of the destination, so every store covers
// whole lines; lane i handles vector tile*64 - lo8 + i, and tile 0 also does
// the <= 3 leading and <= 3 trailing elements.  Scalar path: four elements
// per lane, 64 apart.
template <typename T, int OP, int KIND, bool VEC, bool NT>
__device__ __forceinline__ void seg_tile(T* __restrict__ dst, const T* __restrict__ own, T* __restrict__ dst2,
                                         const T* __restrict__ own2, const T* __restrict__ src, int64_t len,
                                         int64_t e0, int64_t tile, int lane) {
  if constexpr (VEC) {
    int64_t head = (4 - (e0 & 3)) & 3;
    if (head > len) head = len;
    const int64_t nvec = (len - head) >> 2;
    const int64_t tail0 = head + (nvec << 2);
    const int64_t lo8 = (reinterpret_cast<uintptr_t>(dst + head) >> 4) & 7;
    const int64_t v = tile * kWave - lo8 + lane;
    if (v >= 0 && v < nvec) {
      const V4<T> sv = ld4<NT>(reinterpret_cast<const V4<T>*>(src + head) + v);
      if constexpr (KIND == kCopy) {
        st4<NT>(reinterpret_cast<V4<T>*>(dst + head) + v, sv);
      } else {
        const V4<T> ov = ld4<NT>(reinterpret_cast<const V4<T>*>(own + head) + v);
        if constexpr (KIND == kReduce2) {
          const V4<T> o2v = ld4<NT>(reinterpret_cast<const V4<T>*>(own2 + head) + v);
          st4<NT>(reinterpret_cast<V4<T>*>(dst2 + head) + v, comb4<OP>(o2v, sv));
        }
        st4<NT>(reinterpret_cast<V4<T>*>(dst + head) + v, comb4<OP>(ov, sv));
      }
    }
    if (tile == 0) {
      int64_t e = -1;
      if (lane < head) e = lane;
      else if (lane >= 4 && lane - 4 < len - tail0) e = tail0 + (lane - 4);
      if (e >= 0) {
        if constexpr (KIND == kCopy) {
          dst[e] = src[e];
        } else {
          const T s1 = src[e];
          if constexpr (KIND == kReduce2) dst2[e] = comb<OP>(own2[e], s1);
          dst[e] = comb<OP>(own[e], s1);
        }
      }
    }
  } else {
    const int64_t i0 = tile * kTile;
    T sv[4], ov[4], o2v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t e = i0 + u * kWave + lane;
      if (e < len) {
        sv[u] = src[e];
        if constexpr (KIND != kCopy) ov[u] = own[e];
        if constexpr (KIND == kReduce2) o2v[u] = own2[e];
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t e = i0 + u * kWave + lane;
      if (e < len) {
        if constexpr (KIND == kCopy) {
          dst[e] = sv[u];
        } else {
          if constexpr (KIND == kReduce2) dst2[e] = comb<OP>(o2v[u], sv[u]);
          dst[e] = comb<OP>(ov[u], sv[u]);
        }
      }
    }
  }
}

// Wave tile t of the launch -> (rank x, op j, instance, tile within the
// segment); consecutive waves stream consecutive tiles of one block, so a
// workgroup covers 4 KB of each stream and small segments share workgroups.
// The launch has one wave per tile (up to kMaxGrid workgroups).  The
// decomposition is wave-uniform 32-bit scalar arithmetic with precomputed
// divisions, short enough that a wave reaches its loads almost at once:
// with one 16-byte vector per lane in flight, a long prologue would leave
// the memory system idle.
template <typename T, int OP, bool VEC, bool NT, bool XOR>
__global__ __launch_bounds__(kBlock) void step_kernel(const StepArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t wave_in_block = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int32_t P = a.P;
  for (uint32_t t = blockIdx.x * uint32_t(kWavesPerBlock) + wave_in_block; t < a.total_tiles;
       t += gridDim.x * uint32_t(kWavesPerBlock)) {
    const uint32_t seg = fdiv(t, a.tps);
    const uint32_t tile = t - seg * a.tps.d;
    const uint32_t rest = fdiv(seg, a.batch);
    const uint32_t inst = seg - rest * a.batch.d;
    const uint32_t x32 = fdiv(rest, a.ops);
    const int32_t j = int32_t(rest - x32 * a.ops.d);
    const int32_t x = int32_t(x32);
    int ri = 0;
    while (ri + 1 < a.n_ranges && j >= a.ranges[ri + 1].first) ++ri;
    const DevRange& R = a.ranges[ri];
    int32_t p = R.p0 + (j - R.first);  // < 2P
    if (p >= P) p -= P;
    int32_t b, y;
    if constexpr (XOR) {                // t_k(x) = x XOR k: block x XOR p, peer x XOR delta
      b = x ^ p;
      y = x ^ R.delta;
    } else {                            // cyclic: block x - p, peer x + delta (|delta| < P)
      b = x - p;
      if (b < 0) b += P;
      y = x + R.delta;
      if (y >= P) y -= P;
      if (y < 0) y += P;
    }
    const int64_t len = a.q + (b < a.m ? 1 : 0);
    const int64_t off = int64_t(b) * a.q + (b < a.m ? b : a.m);
    const int64_t e0 = int64_t(inst) * a.stride + off;
    T* dst = buf_ptr<T>(a, R.dst, x) + e0;
    const T* src = buf_ptr<T>(a, R.src, y) + e0;
    if (R.kind == kCopy) {
      seg_tile<T, OP, kCopy, VEC, NT>(dst, nullptr, nullptr, nullptr, src, len, e0, tile, lane);
    } else if (R.kind == kReduce) {
      const T* own = buf_ptr<T>(a, R.own, x) + e0;
      seg_tile<T, OP, kReduce, VEC, NT>(dst, own, nullptr, nullptr, src, len, e0, tile, lane);
    } else {
      const T* own = buf_ptr<T>(a, R.own, x) + e0;
      T* dst2 = buf_ptr<T>(a, R.dst2, x) + e0;
      const T* own2 = buf_ptr<T>(a, R.own2, x) + e0;
      seg_tile<T, OP, kReduce2, VEC, NT>(dst, own, dst2, own2, src, len, e0, tile, lane);
    }
  }
}

// Merged runs.  Within one launch, the placements p0 .. p0+count-1 of a
// range share their operation, their buffers and their peer, and rank x's
// blocks at those placements -- x - p (cyclic) or x XOR p (XOR group, for
// an aligned power-of-two range) -- form one run of consecutive blocks,
// wrapping past block P-1 at most once (cyclic).  Peer and own blocks have
// the same index, so the whole run is one elementwise operation over a
// contiguous range of elements per instance, and over the whole row when
// the range covers every placement (every latency-optimal step).  This
// kernel streams each (rank, range) as a flat space of batch * run columns,
// four 4-byte columns per lane (256 per wave tile), so that batches of
// short blocks fill their waves.  The element operations are exactly those
// of step_kernel, only grouped differently.
template <typename T, int OP, int KIND, bool NT>
__device__ __forceinline__ void merged_cols(T* __restrict__ dst, const T* __restrict__ own, T* __restrict__ dst2,
                                            const T* __restrict__ own2, const T* __restrict__ src, const int64_t (&e)[4],
                                            const bool (&live)[4]) {
  T sv[4], ov[4], o2v[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (live[u]) {
      sv[u] = ld1<NT>(src + e[u]);
      if constexpr (KIND != kCopy) ov[u] = ld1<NT>(own + e[u]);
      if constexpr (KIND == kReduce2) o2v[u] = ld1<NT>(own2 + e[u]);
    }
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (live[u]) {
      if constexpr (KIND == kCopy) {
        st1<NT>(dst + e[u], sv[u]);
      } else {
        if constexpr (KIND == kReduce2) st1<NT>(dst2 + e[u], comb<OP>(o2v[u], sv[u]));
        st1<NT>(dst + e[u], comb<OP>(ov[u], sv[u]));
      }
    }
  }
}

template <typename T, int OP, bool NT, bool XOR>
__global__ __launch_bounds__(kBlock) void step_merged_kernel(const StepArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t wave_in_block = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int32_t P = a.P;
  for (uint32_t t = blockIdx.x * uint32_t(kWavesPerBlock) + wave_in_block; t < a.total_tiles;
       t += gridDim.x * uint32_t(kWavesPerBlock)) {
    int ri = 0;
    while (ri + 1 < a.n_ranges && t >= a.tile_first[ri + 1]) ++ri;
    const DevRange& R = a.ranges[ri];
    const uint32_t tr = t - a.tile_first[ri];
    const uint32_t x32 = fdiv(tr, a.tiles[ri]);
    const uint32_t tile = tr - x32 * a.tiles[ri].d;
    const int32_t x = int32_t(x32);
    const bool whole = R.count == P;
    int32_t bf, y;  // first block of rank x's run, peer
    if constexpr (XOR) {
      bf = (x ^ R.p0) & ~(R.count - 1);
      y = x ^ R.delta;
    } else {
      bf = x - R.p0 - R.count + 1;  // > -2P
      if (bf < 0) bf += P;
      if (bf < 0) bf += P;
      y = x + R.delta;
      if (y >= P) y -= P;
      if (y < 0) y += P;
    }
    // elements of the run: from block bf on, count blocks, wrapping at n
    const int64_t off = int64_t(bf) * a.q + (bf < a.m ? bf : a.m);
    const int32_t be = bf + R.count;  // one past the run's last block, <= 2P
    const int32_t bw = be > P ? be - P : be;
    const int64_t off_end = int64_t(bw) * a.q + (bw < a.m ? bw : a.m);
    const int64_t run = be > P ? a.n - off + off_end : off_end - off;
    int64_t e[4];
    bool live[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t g = tile * uint32_t(4 * kWave) + uint32_t(u * kWave + lane);
      const uint32_t inst = fdiv(g, a.run_len[ri]);
      const int64_t v = int64_t(g) - int64_t(inst) * a.run_len[ri].d;
      int64_t i = whole ? v : off + v;
      if (i >= a.n) i -= a.n;
      live[u] = g < a.run_cols[ri] && (whole || v < run);
      e[u] = int64_t(inst) * a.stride + i;
    }
    T* dst = buf_ptr<T>(a, R.dst, x);
    const T* src = buf_ptr<T>(a, R.src, y);
    if (R.kind == kCopy) {
      merged_cols<T, OP, kCopy, NT>(dst, nullptr, nullptr, nullptr, src, e, live);
    } else if (R.kind == kReduce) {
      merged_cols<T, OP, kReduce, NT>(dst, buf_ptr<T>(a, R.own, x), nullptr, nullptr, src, e, live);
    } else {
      merged_cols<T, OP, kReduce2, NT>(dst, buf_ptr<T>(a, R.own, x), buf_ptr<T>(a, R.dst2, x),
                                       buf_ptr<T>(a, R.own2, x), src, e, live);
    }
  }
}

template <typename T, int OP>
int launch_step_t(const StepArgs& a, bool vec, bool nt, int grid, hipStream_t s) {
  // the group is a template argument: the block / peer arithmetic sits in
  // the prologue every wave runs before its first load
  if (a.group == kGroupXor) {
    if (vec && nt) hipLaunchKernelGGL((step_kernel<T, OP, true, true, true>), dim3(grid), dim3(kBlock), 0, s, a);
    else if (vec) hipLaunchKernelGGL((step_kernel<T, OP, true, false, true>), dim3(grid), dim3(kBlock), 0, s, a);
    else hipLaunchKernelGGL((step_kernel<T, OP, false, false, true>), dim3(grid), dim3(kBlock), 0, s, a);
  } else {
    if (vec && nt) hipLaunchKernelGGL((step_kernel<T, OP, true, true, false>), dim3(grid), dim3(kBlock), 0, s, a);
    else if (vec) hipLaunchKernelGGL((step_kernel<T, OP, true, false, false>), dim3(grid), dim3(kBlock), 0, s, a);
    else hipLaunchKernelGGL((step_kernel<T, OP, false, false, false>), dim3(grid), dim3(kBlock), 0, s, a);
  }
  return int(hipGetLastError());
}

}  // namespace

int64_t step_tile_elems() { return kTile; }

int launch_step_merged(const StepArgs& a, int dtype, int op, bool nt, int grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const dim3 g(grid), blk(kBlock);
#define AR_MERGED(T, OP)                                                                                   \
  do {                                                                                                     \
    if (a.group == kGroupXor) {                                                                            \
      if (nt) hipLaunchKernelGGL((step_merged_kernel<T, OP, true, true>), g, blk, 0, s, a);                 \
      else hipLaunchKernelGGL((step_merged_kernel<T, OP, false, true>), g, blk, 0, s, a);                   \
    } else {                                                                                               \
      if (nt) hipLaunchKernelGGL((step_merged_kernel<T, OP, true, false>), g, blk, 0, s, a);                \
      else hipLaunchKernelGGL((step_merged_kernel<T, OP, false, false>), g, blk, 0, s, a);                  \
    }                                                                                                      \
  } while (0)
  if (dtype == 0) {
    if (op == 0) AR_MERGED(int32_t, 0);
    else AR_MERGED(int32_t, 1);
  } else {
    if (op == 0) AR_MERGED(float, 0);
    else AR_MERGED(float, 1);
  }
#undef AR_MERGED
  return int(hipGetLastError());
}

int step_grid(int64_t total_tiles) {
  int64_t blocks = (total_tiles + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks > kMaxGrid) blocks = kMaxGrid;
  if (blocks < 1) blocks = 1;
  return int(blocks);
}

int launch_step(const StepArgs& a, int dtype, int op, bool vec, bool nt, int grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (dtype == 0)
    return op == 0 ? launch_step_t<int32_t, 0>(a, vec, nt, grid, s) : launch_step_t<int32_t, 1>(a, vec, nt, grid, s);
  return op == 0 ? launch_step_t<float, 0>(a, vec, nt, grid, s) : launch_step_t<float, 1>(a, vec, nt, grid, s);
}

}  // namespace ar
