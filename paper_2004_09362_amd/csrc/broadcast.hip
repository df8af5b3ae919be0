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
// Layout and tiles as in fused_col.hpp: one wave per 64 columns of one
// block of one instance, tiles laid on 256-byte boundaries of rank b's
// buffer, ordinary (cached) stores, which streamed faster here than
// nontemporal ones.
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
    const uint32_t seg = fdiv(t, a.tiles);  // seg = instance * P + block
    const uint32_t tile = t - seg * a.tiles.d;
    const uint32_t inst = fdiv(seg, a.pdiv);
    const int32_t b = int32_t(seg - inst * a.pdiv.d);
    const int64_t len = a.q + (b < a.m ? 1 : 0);
    const int64_t e0 = int64_t(inst) * a.stride + int64_t(b) * a.q + (b < a.m ? b : a.m);
    void* const* rot = a.user + b;  // rot[d] is rank (b + d) mod P
    const int64_t lo = ((reinterpret_cast<uintptr_t>(rot[0]) >> 2) + e0) & (kWave - 1);
    const int64_t c = int64_t(tile) * kWave - lo + lane;
    if (c >= 0 && c < len) {
      const int64_t e = e0 + c;
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
