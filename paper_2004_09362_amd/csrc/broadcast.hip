// broadcast.hip -- second half of a split column-fused launch.
//
// For the schedules whose distribution phase hands every rank the same
// result (bandwidth-optimal plans of Sec. 7 in either group, and the Ring of
// Sec. 6), the column kernels can store block b's result on rank b alone;
// this kernel then copies it to ranks b+1, ..., b+P-1.  The copy moves the
// bytes the distribution phase moves, and one more read and write of each
// block than the single fused launch.  It pays at large P: a launch that
// reads P streams and writes P streams at once interleaves reads and writes
// across hundreds of DRAM rows, while a reducing launch (P reads, one
// write) and this one (one read, P - 1 writes) each stream in one
// direction.  On MI355X at P = 127 the pair ran 8% faster than the single
// launch (probes: reducing 6.4 TB/s, broadcasting 5.3 TB/s, fused 5.35
// TB/s).
//
// Layout and tiles as in the reducing launch (col_tile_column,
// device_common.hpp): one wave per 64 columns of one block of one instance,
// tiles laid on 256-byte boundaries of rank b's buffer, or one short block
// of several instances per wave.  After a reducing launch on flat columns
// (a.flat: batches of short blocks) every column's result is on rank 0, and
// the waves take 64 consecutive flat columns each.  Loads and stores are
// nontemporal (NT) or ordinary: from P = 96 ranks, streaming the P - 1
// stores nontemporally at one resident workgroup per CU was 3-4% faster,
// and on flat columns nontemporal stores were 1-11% faster at any P; below
// P = 96 on block tiles, ordinary stores streamed as fast or faster.
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

}  // namespace

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
