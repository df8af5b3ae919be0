// broadcast.hip -- second half of a split column-fused launch.
//
// For the schedules whose distribution phase hands every rank the same
// result (bandwidth-optimal plans of Sec. 7 in either group, and the Ring of
// Sec. 6), the column kernels can store block b's result on rank b alone;
// the broadcast then copies it to ranks b+1, ..., b+P-1.  The copy moves the
// bytes the distribution phase moves, and one more read and write of each
// block than the single fused launch.  It pays at large P: a launch that
// reads P streams and writes P streams at once interleaves reads and writes
// across hundreds of DRAM rows, while a reducing launch (P reads, one
// write) and the broadcast (one read, P - 1 writes) each stream in one
// direction.  On MI355X at P = 127 the pair with the tiled broadcast ran 8%
// faster than the single launch (reducing 6.4 TB/s, broadcasting 5.8 TB/s,
// single launch 5.35 TB/s), and the destination-major broadcast (second
// kernel below, 6.3-6.4 TB/s) gains another 3-4% where it applies.
//
// broadcast_kernel, the tiled copy: layout and tiles as in the reducing
// launch (col_tile_column, device_common.hpp): one wave per 64 columns of
// one block of one instance, tiles laid on 256-byte boundaries of rank b's
// buffer, or one short block of several instances per wave.  After a
// reducing launch on flat columns (a.flat: batches of short blocks) every
// column's result is on rank 0, and the waves take 64 consecutive flat
// columns each.  Loads and stores are nontemporal (NT) or ordinary: from
// P = 96 ranks, streaming the P - 1 stores nontemporally at one resident
// workgroup per CU was 3-4% faster, and on flat columns nontemporal stores
// were 1-11% faster at any P; below P = 96 on block tiles, ordinary stores
// streamed as fast or faster.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "ar_internal.hpp"
#include "device_common.hpp"

namespace ar {

namespace {

template <typename T, bool NT>
__global__ __launch_bounds__(kBlock) void broadcast_kernel(const ColArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t wave_in_block = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int32_t P = a.P;
  for (uint32_t t = blockIdx.x * uint32_t(kWavesPerBlock) + wave_in_block; t < a.total_tiles;
       t += gridDim.x * uint32_t(kWavesPerBlock)) {
    int32_t b = 0;
    int64_t e;
    bool live;
    if (a.flat) {
      const uint32_t g = t * uint32_t(kWave) + uint32_t(lane);
      const uint32_t inst = fdiv(g, a.ndiv);
      e = int64_t(inst) * a.stride + int64_t(g - inst * a.ndiv.d);
      live = g < a.flat_cols;
    } else {
      live = col_tile_column(a, t, lane, b, e);
    }
    void* const* rot = a.user + b;  // rot[d] is rank (b + d) mod P
    if (live) {
      const T v = ld1<NT>(static_cast<const T*>(rot[0]) + e);
#pragma unroll 8
      for (int32_t d = 1; d < P; ++d) st1<NT>(static_cast<T*>(rot[d]) + e, v);
    }
  }
}

// Destination-major copy.  The kernel above writes the P - 1 destinations
// of a column tile at once, so the stores in flight hit P - 1 rank buffers
// (256 MB apart at P = 127, n = 2^26) and HBM writes them at 5.8 TB/s.  Here
// workgroup ids run slice by slice, destination by destination, chunk by
// chunk: the workgroups in flight sweep one destination's buffer in address
// order, and each thread copies 16 bytes once and exits.  A slice's source
// columns are read from HBM once and then from L2 for the other
// destinations: workgroup ids go round-robin over the XCDs, so with C chunks
// per slice a multiple of the XCD count X, workgroup c of a slice runs on
// XCD c mod X for every destination.  The chunk it copies is chunk c
// (interleaved: 1 MB of each slice per XCD, in 4 KB pieces X chunks apart),
// or with a.regions the ((c mod X) * C / X + c / X)-th (XCD x copies the x-th
// contiguous C / X chunks: 256 KB of each slice).  Interleaved chunks stop
// hitting L2 at P = 110-128 below 256 MB per rank (P = 127, 64 MB per rank:
// 36% of the source reads went to HBM), where regions keep them; regions
// also suit blocks on the chunk grid.  With C not a multiple of X the copy
// took 1.3x the time, with 2 MB per XCD 1.4x, and with the index arithmetic
// behind branches (each deferring an argument load, a round trip per
// workgroup) 1.2x.  The chunks of a slice that fall in destination y's own
// block are skipped (y holds that result already), and a chunk holds at most
// two blocks (the host asks for blocks of at least kStreamChunk elements),
// or one root (flat columns).
__device__ __forceinline__ uint32_t sdiv(uint32_t n, const StreamDiv& d) {
  const uint32_t t = __umulhi(n, d.mul);
  return (t + ((n - t) >> d.s1)) >> d.s2;
}

// Root of flat column g: rank 0 on flat columns, else the block of g within
// its instance.  No branches, so that the argument loads are not deferred
// into them (each deferred load is a round trip in every workgroup).
__device__ __forceinline__ uint32_t stream_root(const StreamArgs& a, uint32_t g) {
  const uint32_t i = g - sdiv(g, a.ndiv) * a.n;
  const uint32_t lo = sdiv(i, a.q1div), hi = a.m + sdiv(i - a.big, a.qdiv);
  return a.flat ? 0u : (i < a.big ? lo : hi);
}

// First column after block b0 of the instance holding column `first`
// (block b0 + 1 = P: the instance's end), for block tiles.
__device__ __forceinline__ uint32_t stream_block_end(const StreamArgs& a, uint32_t first, uint32_t b0) {
  const uint32_t i0 = first - sdiv(first, a.ndiv) * a.n;
  return first - i0 + (b0 + 1) * a.q + min(b0 + 1, a.m);
}

// STRADDLE: some block or instance boundary is off the kStreamChunk grid,
// so chunks can span two blocks; such a chunk is copied in whole 16-byte
// groups, each element selected from its root's load (the elements of y's
// own block are rewritten with the value y holds: the same bits).  Without
// STRADDLE only the tail of the column space (and any chunk across a
// boundary, which the host rules out) takes the element path.  Both kinds
// are kept because the instructions on the plain path matter: a workgroup
// does little besides its index arithmetic.  At P = 127, n = 2^26
// (straddles) the element path took 5.37 ms, whole groups 4.82 ms, and whole
// groups behind a separate plain path 4.94 ms; at P = 128 (none) the kernel
// with the plain path first took 4.64 ms and the whole-group one 4.80 ms.
template <bool NT, bool STRADDLE>
__global__ __launch_bounds__(kStreamBlock) void broadcast_stream_kernel(const StreamArgs a) {
  const uint32_t id = a.id0 + blockIdx.x;
  const uint32_t s = sdiv(id, a.sdiv);
  const uint32_t r = id - s * a.sdiv.d;
  const uint32_t y = sdiv(r, a.cdiv);
  uint32_t c = r - y * a.cdiv.d;  // workgroup c of the slice runs on XCD c mod X
  if (a.regions) c = (c & ((1u << a.xcd_shift) - 1u)) * a.per_xcd + (c >> a.xcd_shift);
  const uint32_t chunk = s * a.cdiv.d + c;
  const uint32_t first = chunk * kStreamChunk;
  const uint32_t last = min(first + kStreamChunk, a.cols) - 1;
  const uint32_t b0 = stream_root(a, first), b1 = stream_root(a, last);
  if (chunk >= a.chunks || (b0 == y && b1 == y)) return;
  const uint32_t g = first + threadIdx.x * 4u;
  int32_t* dst = static_cast<int32_t*>(a.user[y]);
  const int32_t* s0 = static_cast<const int32_t*>(a.user[b0]);
  if constexpr (STRADDLE) {
    if (first + kStreamChunk <= a.cols) {
      i32x4 v = *reinterpret_cast<const i32x4*>(s0 + g);
      if (b0 != b1) {  // block b0 ends at column bnd of this chunk
        const int32_t* s1 = static_cast<const int32_t*>(a.user[b1]);
        const i32x4 w = *reinterpret_cast<const i32x4*>(s1 + g);
        const uint32_t bnd = stream_block_end(a, first, b0);
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = g + uint32_t(i) < bnd ? v[i] : w[i];
      }
      if constexpr (NT) __builtin_nontemporal_store(v, reinterpret_cast<i32x4*>(dst + g));
      else *reinterpret_cast<i32x4*>(dst + g) = v;
      return;
    }
  } else {
    if (b0 == b1 && first + kStreamChunk <= a.cols) {
      const i32x4 v = *reinterpret_cast<const i32x4*>(s0 + g);
      if constexpr (NT) __builtin_nontemporal_store(v, reinterpret_cast<i32x4*>(dst + g));
      else *reinterpret_cast<i32x4*>(dst + g) = v;
      return;
    }
  }
  // the chunk at the end of the column space (and, without STRADDLE, any
  // chunk across a boundary): element by element
  const int32_t* s1 = static_cast<const int32_t*>(a.user[b1]);
  const uint32_t bnd = a.flat ? a.cols : stream_block_end(a, first, b0);
  const bool w0 = b0 != y, w1 = b1 != y;
#pragma unroll
  for (uint32_t i = 0; i < 4; ++i) {
    const uint32_t gi = g + i;
    const bool lo = gi < bnd;
    if (gi < a.cols && (lo ? w0 : w1)) st1<NT>(dst + gi, (lo ? s0 : s1)[gi]);
  }
}

}  // namespace

int launch_broadcast_stream(const StreamArgs& a, bool nt, bool straddle, uint32_t grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const dim3 g(grid), blk(kStreamBlock);
  if (straddle) {
    if (nt) hipLaunchKernelGGL((broadcast_stream_kernel<true, true>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((broadcast_stream_kernel<false, true>), g, blk, 0, s, a);
  } else {
    if (nt) hipLaunchKernelGGL((broadcast_stream_kernel<true, false>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((broadcast_stream_kernel<false, false>), g, blk, 0, s, a);
  }
  return int(hipGetLastError());
}

int launch_broadcast(const ColArgs& a, int dtype, bool nt, int grid, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const dim3 g(grid), blk(kBlock);
  if (dtype == 0) {
    if (nt) hipLaunchKernelGGL((broadcast_kernel<int32_t, true>), g, blk, a.lds, s, a);
    else hipLaunchKernelGGL((broadcast_kernel<int32_t, false>), g, blk, a.lds, s, a);
  } else {
    if (nt) hipLaunchKernelGGL((broadcast_kernel<float, true>), g, blk, a.lds, s, a);
    else hipLaunchKernelGGL((broadcast_kernel<float, false>), g, blk, a.lds, s, a);
  }
  return int(hipGetLastError());
}

}  // namespace ar
