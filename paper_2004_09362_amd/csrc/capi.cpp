// capi.cpp -- the C ABI of libar.so (declared in include/ar.h).
//
// Argument checking, workspace management and launch orchestration.  The
// schedule comes from plan.cpp, the kernels from kernels.hip (step),
// fused_lo.hip, fused_col.hpp (instantiated per P in units that build.py
// writes), fused_group.hip and
// broadcast.hip; nothing here computes on the host.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <array>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/ar.h"
#include "ar_internal.hpp"

// Step launches moving at least this many bytes use nontemporal loads and
// stores; the fused kernels, whose many concurrent streams gain from it at
// smaller sizes, switch at a lower mark.
constexpr int64_t kNtThresholdBytes = int64_t(512) << 20;
constexpr int64_t kFusedNtThresholdBytes = int64_t(128) << 20;
// Plans whose ranks all receive the same result (bandwidth-optimal in either
// group, the Ring) run fused as a reducing launch plus a broadcast from this
// many ranks up (broadcast.hip): measured faster at P = 64 and 127, slower
// at P = 24 and 48 (with the tiled broadcast).  Block-tiled plans whose
// instance spans kSplitMidMinBytes per rank split from kSplitMidMinP ranks:
// with the current destination-major broadcast whole calls took 5-9% less
// time than the single launch at P = 24 and 28 with 32-128 MB per rank (the
// gradient-sync shape, P = 24 at 64 MB: 7%; its Ring: 6%), 1% less at P = 16
// (64 MB); the pair's launches summed to 5-11% less at P = 32-56 with 64 MB,
// and at 16 MB from 9% less to 5% more.
constexpr int32_t kSplitMinP = 64;
constexpr int32_t kSplitMidMinP = 24;
constexpr int64_t kSplitMidMinBytes = int64_t(32) << 20;
// Flat short-block sums in the rank-slot kernel (not the XOR group's) split
// from this many ranks up: their single launch streams 5.0-5.6 TB/s there and
// the pair up to 6.0 (P = 37: 7%, P = 48: 15% faster with caps 4 and 2 and a
// nontemporal broadcast; P = 24 even; the Ring at P = 24 and the XOR kernel
// at P = 32 slower).
constexpr int32_t kFlatSplitMinP = 33;
// From this many ranks up the broadcast streams its P - 1 stores
// nontemporally (at kFusedNtThresholdBytes and above) with one workgroup per
// CU: 3-4% faster at P = 100-128 than cached stores at two workgroups per CU,
// the same at P = 64, and 13% slower at P = 48.  Neither change helps alone.
constexpr int32_t kBcastStreamMinP = 96;
// The destination-major broadcast (broadcast.hip) by default: on flat
// columns at any P, and on block tiles where a rank's span of the call
// reaches kBcastStreamMinBytes (smaller spans not measured).  Measured
// against the tiled copy (rank rows back to back), it took 6-24% less time
// on block tiles at P = 64-128 and 2-256 MB per rank (5.7-7.2 TB/s against
// 5.0-6.2), and 6-21% less on flat columns at P = 37-128 and 4.5-72 MB per
// rank.  Its chunk order: XCD regions on flat columns above
// kBcastFlatInterleaveMaxBytes per rank (interleaved up to it, where short
// slices left XCDs idle, and at exactly 16 MiB, two full slices, 1-5% less
// time than regions at P = 37-127; regions 1-4% less at 20, 28 and 32 MiB,
// within 2% either way at 24 MiB and above), and on block tiles whose
// blocks all start on the chunk grid from kBcastRegionMinP ranks or from
// kBcastAlignedRegionMinBytes per rank (P = 128 at 8-32 MiB: 35-38% less
// time than interleaved; P = 64 at 32-256 MiB and P = 32 at 64 MiB: 3-5%
// less; P = 16-64 at 8-16 MiB: 1-8% more, so interleaved there); with
// straddling chunks interleaved below kBcastRegionMinP ranks (P = 100:
// 5-10% less time than regions) or from kBcastInterleaveMinBytes per rank
// (P = 127 at 256 MB: 5%), and regions otherwise, where the interleaved
// chunks read their sources from L2 no more (P = 127 below 256 MB per rank:
// 1.1-2.0x the time of regions).
constexpr int64_t kBcastStreamMinBytes = int64_t(2) << 20;
constexpr int64_t kBcastFlatInterleaveMaxBytes = int64_t(16) << 20;
constexpr int64_t kBcastInterleaveMinBytes = int64_t(256) << 20;
constexpr int64_t kBcastAlignedRegionMinBytes = int64_t(32) << 20;
constexpr int32_t kBcastRegionMinP = 104;
// Blocks of at most this many elements (many small instances) are packed:
// a column-fused wave takes one block of 64 / max_len instances instead of 64
// columns of one block of one instance, laid on 256-byte boundaries (which
// split a short block over two waves).  Measured against blocked tiles:
// 1.5-1.9x at P = 127 and 12 with blocks of 8-19 elements, 1.3x with
// blocks of 33, 1.6x for the Ring at P = 24; within 4% of them for
// bandwidth-optimal P = 24 and shifted P = 37 with blocks of 4-9.
constexpr int64_t kPackMaxLen = 64;
// Shifted sums (0 < r < L) on long blocks take the rank-slot kernel at odd P
// from this many ranks: there the block-tiled shifted kernel holds all P
// starred sums at one wave per SIMD (256 VGPRs plus 24-153 AGPRs), the
// rank-slot kernel, which keeps only the sums its r needs, two.  Measured on
// n = 2^24-2^26 fp32: 1-10% less time at P = 99, 111, 125 and 127 (the large
// workload at k = 10: 5%), within 2.4% either way at P = 87, 3-9% more at
// P = 33-81 (odd or even) and 1-5% more at even P = 72-100; mixed at P = 120
// and faster at P = 128 (its kernel at three waves) by 3-5%.  Also at
// P = kRotShiftedSmallMinP-kRotShiftedSmallMaxP with instances of at most
// kRotShiftedSmallMaxBytes per rank: 1-5% less time at P = 24, 33, 34, 37,
// 47 and 48 with 8-32 MB per rank (the prime_sweep shape, P = 37 at 16 MB:
// 4-5% at k = 7-11), 1-10% more at 64 MB; at P = 64-93 within 2.4% either
// way up to 32 MB.  Shifted max plans take this second rule as well (their
// rank-slot kernels exist at P = 24-48 only): 4-7% less time at P = 37 and
// 48 with 16 MB per rank, 2.6% more at P = 24 with 32 MB.
constexpr int32_t kRotShiftedMinP = 97;
constexpr int32_t kRotShiftedSmallMinP = 24, kRotShiftedSmallMaxP = 48;
constexpr int64_t kRotShiftedSmallMaxBytes = int64_t(32) << 20;
// Plans whose ranks all receive one result (bandwidth-optimal, the Ring)
// take the rank-slot kernel on long blocks too where it splits (from
// kFlatSplitMinP ranks: the reducing launch stores to rank 0, the flat
// broadcast copies) and below kRotOneMaxBytes per rank instance.  Against
// the block-tiled kernels (split from P = 32 at 64 MiB and from P = 64),
// sums and max took 3-9% less time at P = 37 and 127 with 16-128 MB per
// rank (the Ring at P = 127: 3-5%), within 1.7% either way at P = 64-100;
// at 256 MB (P = 127) 0.7% more.  Unsplit, at P = 8-32, the two were
// within 4% either way with no consistent sign (the gradient-sync shape,
// P = 24 at 64 MB: 4% more), so those keep block tiles.
constexpr int32_t kRotOneMinP = 33;
// The XOR group's plans run on flat columns on long blocks as well
// (Recursive Halving and the hybrids; Recursive Doubling, r = L, keeps block
// tiles: 1% faster for sums and 14% for max at P = 32).  Sums, whose flat
// kernel leaves the block out, took 1-7% less time at P = 8-128 with
// 16-64 MB per rank (P = 32 hybrids: 4%; P = 128 at 16 MB, split: 7%), max,
// whose flat kernel orders each pair by the lane's block, 0-6% less; the
// same or better at every shape measured.
constexpr int64_t kRotOneMaxBytes = int64_t(256) << 20;
// Step launches whose blocks hold at most this many elements stream each
// range's run of blocks as one flat space per rank (step_merged_kernel):
// short blocks otherwise leave most lanes of the 1 KB block tiles idle.
// Measured at P = 24 and 127: merged runs 2.1x faster with blocks of 64
// elements, 4-12% with 128-256; block tiles (16-byte lanes) 9-20% faster
// from 512 on.
constexpr int64_t kMergeMaxLen = 256;

// Occupancy caps of the fused kernels.  Every fused launch streams P rank
// buffers in and out at once, and HBM serves that pattern faster when fewer
// waves are resident: fewer DRAM rows are open at a time.  A launch caps the
// workgroups resident per CU (one wave per SIMD each) by reserving LDS it
// does not use.  The caps below are the best points measured on MI355X
// (gfx950) at the benchmark shapes, against no cap:
//   latency-optimal, 65536 instances of 106 elements: P = 5 and 7 at 5,
//     P = 6 at 4, P = 12 at 3-4 (2-4%);
//   bandwidth-optimal, P = 24 and 32 at 3-4, P = 37 at 3 (3-4%);
//   shifted, P = 37 at 2-3 (2%); at P = 127 its registers already allow only
//     one wave per SIMD, and a cap changes nothing;
//   the Ring at P = 24: 4 (2%);
//   split launches (P = 127): the reducing launch at 3-6, the broadcast at 2
//     (1 with nontemporal stores, from kBcastStreamMinP ranks up); the
//     rank-slot kernel's reducing launch below kSplitMinP ranks at 4;
//   block-tiled launches of every kind up to P = 8: none up to P = 6, 6 at
//     P = 7-8 (large messages: P = 2 4.45 against 2.80 TB/s at the former
//     cap of 4, P = 4 6.06 against 4.56, shifted P = 4 6.17 against 3.88);
//   flat columns for short blocks (fused_flat): none up to P = 6 (a cap of 4
//     cost 10-29% there), P = 7-8 at 6, P = 12 at 3-4, P = 24, 32 and 37 at 2
//     (3-7%); none from P = 64 (caps of 1-4 the same or slower).
// AR_FUSED_CAP = N (both launches) or N,M (fused launch, broadcast) overrides
// them; 0 is no cap.
static int32_t lo_cap(int32_t P) { return P <= 4 ? 0 : P == 6 ? 4 : P <= 7 ? 5 : P <= 11 ? 4 : 3; }

// Which kernel runs a plan on the FUSED path: the latency-optimal kernel for
// P <= 16 (flat columns, no block index), the column kernels of the cyclic
// butterfly schedules (tiled by block; flat columns when r = L), or the
// column kernels of the XOR group and of the Ring.  Where every rank
// receives the same result a broadcast launch may follow (fused_split).
enum FusedKind { kFusedNone = 0, kFusedLo = 1, kFusedCol = 2, kFusedXor = 3, kFusedRing = 4 };

struct ar_plan {
  ar::Schedule s;
  int32_t dtype = 0, op = 0;
  // Tuning overrides read from the environment at plan creation:
  // AR_STEP_NT / AR_FUSED_NT = 0|1 (nontemporal never / always; default by
  // launch size),
  // AR_FUSED_SPLIT = 0|1 (single fused launch / reduce plus broadcast, where
  // every rank receives the same result; default by P), AR_BCAST_NT = 0|1
  // (the broadcast's loads and stores; default by P and launch size),
  // AR_BCAST_STREAM = 0|1|2|3 (the broadcast tiled by block / destination by
  // destination wherever the call allows it, with the chunk order by size,
  // interleaved, or in XCD regions; default by the size rules at
  // kBcastStreamMinBytes, kBcastFlatInterleaveMaxBytes, kBcastInterleaveMinBytes,
  // kBcastAlignedRegionMinBytes and kBcastRegionMinP),
  // AR_FUSED_PACKED = 0|1 (column tiles of one block of one instance / of
  // several instances, for blocks of up to 64 elements; default: packed for
  // batches whose blocks hold up to kPackMaxLen elements), AR_FUSED_ROTATE =
  // 0|1 (flat columns for sums other than the latency-optimal ones -- the
  // rank-slot kernel, or the XOR kernel without the block: never / always;
  // default: for blocks of up to kPackMaxLen elements), AR_STEP_MERGE = 0|1
  // (step launches as merged runs of blocks: never / wherever the ranges
  // allow; default: for blocks of up to kMergeMaxLen elements).
  int32_t nt_mode = -1, fused_nt_mode = -1, split_mode = -1, bcast_nt_mode = -1, bcast_stream_mode = -1;
  int32_t packed_mode = -1, rotate_mode = -1, merge_mode = -1;
  bool fused_split = false;
  // Sums whose blocks hold at most kPackMaxLen elements run on flat columns
  // whenever the batch's columns fit in 32 bits: the cyclic butterfly plans
  // with r < L and the Ring in the rank-slot kernel, the XOR group's plans
  // in its own kernel with the block left out.  Split there, the reducing
  // launch stores every column's result on rank 0 and the broadcast copies
  // it to the others.
  bool fused_flat = false;
  // Occupancy caps (resident workgroups per CU; 0: none) of the fused launch
  // and of the broadcast that follows a split one (AR_FUSED_CAP overrides).
  int32_t fused_cap = 0, bcast_cap = 0;
  int32_t path = AR_PATH_AUTO;
  int32_t fused_kind = kFusedNone;
  bool fused_ok = false;
  void* scratch = nullptr;
  size_t scratch_bytes = 0;
  int scratch_device = -1;
  // Scratch buffers replaced by larger ones, with their devices: kept until
  // ar_plan_destroy, since graphs captured earlier may still address them.
  std::vector<std::pair<void*, int>> retired;
  hipStream_t last_stream = nullptr;
  bool ran = false;
};

namespace ar {

// Column-fused kernels of the cyclic butterfly schedules: one instantiation
// per P (units that build.py writes), bandwidth-optimal (r = 0) or shifted
// (r >= 1).
int launch_fused_col_any(const ColArgs& a, int P, int dtype, int op, bool nt, int grid, void* stream) {
  switch (P) {
#define AR_BO_CASE(PP)                                                                                \
  case PP:                                                                                            \
    return a.r == 0 ? launch_fused_bo<PP>(a, dtype, op, nt, grid, stream)                             \
                    : launch_fused_mid<PP>(a, dtype, op, nt, grid, stream);
#define AR_BO_CASE8(B) AR_BO_CASE(B) AR_BO_CASE(B + 1) AR_BO_CASE(B + 2) AR_BO_CASE(B + 3) \
  AR_BO_CASE(B + 4) AR_BO_CASE(B + 5) AR_BO_CASE(B + 6) AR_BO_CASE(B + 7)
    AR_BO_CASE8(2) AR_BO_CASE8(10) AR_BO_CASE8(18) AR_BO_CASE8(26) AR_BO_CASE8(34) AR_BO_CASE8(42)
    AR_BO_CASE8(50) AR_BO_CASE8(58) AR_BO_CASE8(66) AR_BO_CASE8(74) AR_BO_CASE8(82) AR_BO_CASE8(90)
    AR_BO_CASE8(98) AR_BO_CASE8(106) AR_BO_CASE8(114) AR_BO_CASE(122) AR_BO_CASE(123) AR_BO_CASE(124)
    AR_BO_CASE(125) AR_BO_CASE(126) AR_BO_CASE(127) AR_BO_CASE(128)
#undef AR_BO_CASE8
#undef AR_BO_CASE
    default: return int(hipErrorInvalidValue);
  }
}

int launch_fused_rot_any(const ColArgs& a, int P, int dtype, int op, bool ring, int grid, void* stream) {
  switch (P) {
#define AR_ROT_CASE(PP) \
  case PP: return launch_fused_rot<PP>(a, dtype, op, ring, grid, stream);
#define AR_ROT_CASE8(B) AR_ROT_CASE(B) AR_ROT_CASE(B + 1) AR_ROT_CASE(B + 2) AR_ROT_CASE(B + 3) \
  AR_ROT_CASE(B + 4) AR_ROT_CASE(B + 5) AR_ROT_CASE(B + 6) AR_ROT_CASE(B + 7)
    AR_ROT_CASE8(2) AR_ROT_CASE8(10) AR_ROT_CASE8(18) AR_ROT_CASE8(26) AR_ROT_CASE8(34) AR_ROT_CASE8(42)
    AR_ROT_CASE8(50) AR_ROT_CASE8(58) AR_ROT_CASE8(66) AR_ROT_CASE8(74) AR_ROT_CASE8(82) AR_ROT_CASE8(90)
    AR_ROT_CASE8(98) AR_ROT_CASE8(106) AR_ROT_CASE8(114) AR_ROT_CASE(122) AR_ROT_CASE(123) AR_ROT_CASE(124)
    AR_ROT_CASE(125) AR_ROT_CASE(126) AR_ROT_CASE(127) AR_ROT_CASE(128)
#undef AR_ROT_CASE8
#undef AR_ROT_CASE
    default: return int(hipErrorInvalidValue);
  }
}

}  // namespace ar

namespace {

thread_local std::string g_err;

ar_status fail(ar_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

ar_status hip_fail(hipError_t e, const char* what) {
  g_err = std::string(what) + ": " + hipGetErrorString(e);
  return AR_ERR_HIP;
}

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// Check the table of rank pointers: non-null, 4-byte aligned, no overlap.
// Returns AR_OK and whether every buffer is 16-byte aligned.
ar_status check_buffers(const ar_plan* pl, void* const* bufs, int64_t batch, int64_t stride, bool* all16) {
  const int32_t P = pl->s.P;
  const int64_t extent = ((batch - 1) * stride + pl->s.n) * 4;
  // on the stack (P <= 128): the allocation-free entry point uses this too
  std::array<std::pair<uintptr_t, int32_t>, ar::kMaxP> sorted;
  *all16 = true;
  for (int32_t x = 0; x < P; ++x) {
    const uintptr_t p = reinterpret_cast<uintptr_t>(bufs[x]);
    if (p == 0) return fail(AR_ERR_INVALID_ARG, "rank buffer " + std::to_string(x) + " is NULL");
    if (p % 4 != 0) return fail(AR_ERR_INVALID_ARG, "rank buffer " + std::to_string(x) + " is not 4-byte aligned");
    if (p % 16 != 0) *all16 = false;
    sorted[size_t(x)] = {p, x};
  }
  std::sort(sorted.begin(), sorted.begin() + P);
  for (size_t i = 1; i < size_t(P); ++i)
    if (extent > 0 && sorted[i].first < sorted[i - 1].first + uintptr_t(extent))
      return fail(AR_ERR_ALIAS, "rank buffers " + std::to_string(sorted[i - 1].second) + " and " +
                                    std::to_string(sorted[i].second) + " overlap");
  return AR_OK;
}

ar_status ensure_scratch(ar_plan* pl, size_t need, int device, hipStream_t stream) {
  if (pl->scratch && pl->scratch_bytes >= need && pl->scratch_device == device) return AR_OK;
  // An allocation cannot be captured into a graph: refuse it there (the call
  // is then not enqueued) rather than fail the capture.
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cap) != hipSuccess) {
    (void)hipGetLastError();
    cap = hipStreamCaptureStatusNone;
  }
  if (cap != hipStreamCaptureStatusNone)
    return fail(AR_ERR_UNSUPPORTED, "the plan needs " + std::to_string(need) +
                                        " bytes of scratch, which cannot be allocated while the stream is captured; "
                                        "run one call with this device, batch and stride before capturing");
  // Growth on the same device at least doubles the buffer, so that the
  // buffers kept until destroy (below) add up to less than twice the last;
  // if the doubled size cannot be had, exactly the need.
  size_t want = need;
  if (pl->scratch && pl->scratch_device == device) want = std::max(need, pl->scratch_bytes * 2);
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, want);
  if (e != hipSuccess && want > need) {
    (void)hipGetLastError();
    want = need;
    e = hipMalloc(&p, want);
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(AR_ERR_OUT_OF_MEMORY, "scratch of " + std::to_string(need) + " bytes: " + hipGetErrorString(e));
  }
  // the old buffer stays allocated until ar_plan_destroy: work already
  // enqueued, and graphs captured earlier, may still use it
  if (pl->scratch) pl->retired.push_back({pl->scratch, pl->scratch_device});
  pl->scratch = p;
  pl->scratch_bytes = want;
  pl->scratch_device = device;
  return AR_OK;
}

// LDS a workgroup reserves so that at most `cap` workgroups fit on a CU of
// `device` (0 for no cap, or when the device allows no such reservation).
// The device's LDS sizes are cached per device; threads that query the same
// device at once store the same values.
uint32_t cap_lds(int32_t cap, int device) {
  static std::atomic<int64_t> per_cu[64], per_block[64];
  if (cap <= 0 || device < 0 || device >= 64) return 0;
  int64_t cu = per_cu[device].load(std::memory_order_acquire);
  int64_t blk = per_block[device].load(std::memory_order_acquire);
  if (cu == 0 || blk == 0) {
    int a = 0, b = 0;
    if (hipDeviceGetAttribute(&a, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, device) != hipSuccess ||
        hipDeviceGetAttribute(&b, hipDeviceAttributeMaxSharedMemoryPerBlock, device) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    cu = a;
    blk = b;
    per_block[device].store(blk, std::memory_order_release);
    per_cu[device].store(cu, std::memory_order_release);
  }
  // cap workgroups fit, cap + 1 do not (1 KB margin, 512-byte allocation
  // steps); a reservation above the per-workgroup limit cannot enforce it
  const int64_t bytes = (cu / cap - 1024) / 512 * 512;
  if (bytes <= 0 || cu / (cap + 1) >= bytes || bytes > blk) return 0;
  return uint32_t(bytes);
}

// Chunks per slice of the destination-major broadcast on `device`: 256
// chunks (1 MB) per XCD, times the XCD count, taken as the CU count over the
// 32 CUs of a gfx950 XCD (8 on a whole MI355X, fewer on a partition).  The
// CU count is cached per device like the LDS sizes above.
uint32_t stream_slice_chunks(int device) {
  static std::atomic<int32_t> cus[64];
  int32_t c = (device >= 0 && device < 64) ? cus[device].load(std::memory_order_acquire) : 0;
  if (c == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || v <= 0) {
      (void)hipGetLastError();
      v = 32;
    }
    c = v;
    if (device >= 0 && device < 64) cus[device].store(c, std::memory_order_release);
  }
  return 256u * uint32_t(std::max<int32_t>(1, c / 32));
}

// Arguments of the destination-major broadcast (broadcast.hip) when the
// call allows it: instances contiguous (batch 1 or stride n), every rank
// buffer 16-byte aligned, the column space and the grid within 32-bit
// counts, and on block tiles blocks of at least kStreamChunk elements (a
// chunk then spans at most two roots).  False: the tiled broadcast runs.
bool stream_bcast_args(const ar_plan* pl, void* const* bufs, int64_t batch, int64_t stride, bool flat, bool regions,
                       int device, ar::StreamArgs* sa) {
  const ar::Schedule& s = pl->s;
  if (batch > 1 && stride != s.n) return false;
  const int64_t cols = batch * s.n;
  if (cols < 1 || cols > int64_t(UINT32_MAX) - ar::kStreamChunk) return false;
  if (!flat && s.n / s.P < int64_t(ar::kStreamChunk)) return false;
  for (int32_t x = 0; x < s.P; ++x)
    if (reinterpret_cast<uintptr_t>(bufs[x]) % 16 != 0) return false;
  // chunks per slice: at most 1 MB per XCD interleaved, 256 KB per XCD in
  // regions (at 8-32 MB per rank 1 MB regions ran 3-50% slower; from 64 MB
  // the sizes ran within a few percent), evened out over the slices and
  // rounded up to the XCD count, so that the last slice is about as full as
  // the others (a short last slice in regions leaves most XCDs idle)
  const uint32_t xcds = stream_slice_chunks(device) / 256;
  uint32_t shift = 0;
  while ((1u << shift) < xcds) ++shift;
  const bool reg = regions && (1u << shift) == xcds;
  const uint32_t chunks = uint32_t((cols + ar::kStreamChunk - 1) / ar::kStreamChunk);
  const uint32_t cmax = (reg ? 64u : 256u) * xcds;
  const uint32_t slices = (chunks + cmax - 1) / cmax;
  const uint32_t C = ((chunks + slices - 1) / slices + xcds - 1) / xcds * xcds;
  const int64_t grid = (int64_t(chunks) + C - 1) / C * C * s.P;
  if (grid > int64_t(UINT32_MAX) / ar::kStreamBlock) return false;  // work-items per launch below 2^32
  std::memset(sa, 0, sizeof *sa);
  for (int32_t x = 0; x < s.P; ++x) sa->user[x] = bufs[x];
  sa->P = uint32_t(s.P);
  sa->cols = uint32_t(cols);
  sa->n = uint32_t(s.n);
  sa->q = uint32_t(s.n / s.P);
  sa->m = uint32_t(s.n % s.P);
  sa->big = sa->m * (sa->q + 1);
  sa->flat = flat ? 1 : 0;
  sa->ndiv = ar::stream_div(uint32_t(s.n));
  sa->q1div = ar::stream_div(sa->q + 1);
  sa->qdiv = ar::stream_div(std::max<uint32_t>(sa->q, 1));
  sa->cdiv = ar::stream_div(C);
  sa->sdiv = ar::stream_div(C * uint32_t(s.P));
  sa->chunks = chunks;
  sa->id0 = 0;
  sa->regions = reg ? 1 : 0;
  sa->xcd_shift = shift;
  sa->per_xcd = C / xcds;
  return true;
}

bool use_nt(int32_t mode, int64_t bytes, int64_t threshold = kNtThresholdBytes) {
  return mode == 1 || (mode < 0 && bytes >= threshold);
}

// Timing-only HIP events (no system-scope fence) recorded on the launch
// stream before the first launch of an execute and after each launch
// (ar_execute_timed).  The first failure is kept; the events are destroyed
// with the timer.
struct LaunchTimer {
  hipStream_t stream = nullptr;
  std::vector<hipEvent_t> ev;
  hipError_t err = hipSuccess;
  void mark() {
    if (err != hipSuccess) return;
    hipEvent_t e = nullptr;
    hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
    if (r == hipSuccess) {
      ev.push_back(e);
      r = hipEventRecord(e, stream);
    }
    if (r != hipSuccess) err = r;
  }
  ~LaunchTimer() {
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
  }
  LaunchTimer() = default;
  LaunchTimer(const LaunchTimer&) = delete;
  LaunchTimer& operator=(const LaunchTimer&) = delete;
};

ar_status run_stepwise(ar_plan* pl, void* const* bufs, int64_t batch, int64_t stride, bool vec, hipStream_t stream,
                       int device, LaunchTimer* tm, bool noalloc) {
  const ar::Schedule& s = pl->s;
  ar::StepArgs a;
  std::memset(&a, 0, sizeof a);
  for (int32_t x = 0; x < s.P; ++x) a.user[x] = bufs[x];
  a.P = s.P;
  a.group = s.group;
  a.n = s.n;
  a.stride = stride;
  a.q = s.n / s.P;
  a.m = s.n % s.P;
  if (s.uses_scratch) {
    // Scratch mirrors the caller's layout (same element index, same 16-byte
    // phase), one region per rank, X then Y.
    const int64_t rank_stride = round_up((batch - 1) * stride + s.n, 64);
    const size_t need = size_t(2) * s.P * size_t(rank_stride) * 4;
    char* base = nullptr;
    if (noalloc) {
      // the device's file-scope array (noalloc.hip), never an allocation
      if (need > size_t(ar::kNoAllocScratchBytes))
        return fail(AR_ERR_UNSUPPORTED, "the call needs " + std::to_string(need) +
                                            " bytes of scratch; ar_execute_noalloc holds at most " +
                                            std::to_string(ar::kNoAllocScratchBytes));
      void* p = nullptr;
      const int e = ar::noalloc_scratch(device, &p);
      if (e != 0) return hip_fail(hipError_t(e), "hipGetSymbolAddress(scratch)");
      base = static_cast<char*>(p);
    } else {
      ar_status st = ensure_scratch(pl, need, device, stream);
      if (st != AR_OK) return st;
      base = static_cast<char*>(pl->scratch);
    }
    a.scratch_rank_stride = rank_stride;
    a.scratch[0] = base;
    a.scratch[1] = base + size_t(s.P) * size_t(rank_stride) * 4;
  }
  const int64_t max_len = a.q + (a.m ? 1 : 0);
  const int64_t tile = ar::step_tile_elems();
  // +32: a tile grid shifted onto 128-byte lines may need one more tile
  const int64_t tps = std::max<int64_t>(1, (max_len + 32 + tile - 1) / tile);
  a.tps = ar::make_fastdiv(uint32_t(std::min<int64_t>(tps, INT32_MAX)));
  a.batch = ar::make_fastdiv(uint32_t(std::min<int64_t>(batch, INT32_MAX)));
  if (tm) tm->mark();
  for (const ar::Launch& l : s.launches) {
    a.n_ranges = int32_t(l.ranges.size());
    int32_t first = 0;
    for (int32_t i = 0; i < a.n_ranges; ++i) {
      const ar::Range& r = l.ranges[i];
      a.ranges[i] = ar::DevRange{r.p0, r.count, r.kind, r.delta, r.dst, r.own, r.dst2, r.own2, r.src, first};
      first += r.count;
    }
    a.ops = ar::make_fastdiv(uint32_t(first));
    // Nontemporal accesses for launches that stream far more than the
    // Infinity Cache holds; smaller ones keep their output cached for the
    // next step, which reads it.
    int64_t blocks_touched = 0;
    for (const ar::Range& r : l.ranges) blocks_touched += int64_t(r.count) * (r.kind == ar::kCopy ? 2 : r.kind == ar::kReduce ? 3 : 5);
    const int64_t launch_bytes = blocks_touched * s.n * batch * 4;
    const bool nt = use_nt(pl->nt_mode, launch_bytes);
    // Merged runs: every range's blocks of a rank must form one run (always
    // in the cyclic group; aligned power-of-two ranges in the XOR group).
    bool merge = pl->merge_mode == 1 || (pl->merge_mode < 0 && max_len <= kMergeMaxLen);
    for (const ar::Range& r : l.ranges)
      if (s.group == ar::kGroupXor && ((r.count & (r.count - 1)) != 0 || r.p0 % r.count != 0)) merge = false;
    if (merge) {
      int64_t total = 0;
      for (int32_t i = 0; i < a.n_ranges && merge; ++i) {
        const ar::Range& r = l.ranges[i];
        const int64_t run = r.count == s.P ? s.n : int64_t(r.count) * max_len;
        const int64_t cols = batch * run;
        const int64_t tiles = (cols + 255) / 256;
        if (cols >= (int64_t(1) << 32) - 256) {
          merge = false;
          break;
        }
        a.run_len[i] = ar::make_fastdiv(uint32_t(run));
        a.run_cols[i] = uint32_t(cols);
        a.tiles[i] = ar::make_fastdiv(uint32_t(tiles));
        a.tile_first[i] = uint32_t(std::min<int64_t>(total, INT32_MAX));
        total += int64_t(s.P) * tiles;
      }
      if (merge && total < (int64_t(1) << 31)) {
        a.total_tiles = uint32_t(total);
        const int e = ar::launch_step_merged(a, pl->dtype, pl->op, nt, ar::step_grid(total), stream);
        if (e != 0) return hip_fail(hipError_t(e), "merged step kernel launch");
        if (tm) tm->mark();
        continue;
      }
    }
    const int64_t total_tiles = int64_t(s.P) * first * batch * tps;
    if (total_tiles >= (int64_t(1) << 31))
      return fail(AR_ERR_UNSUPPORTED, "one step would need 2^31 or more tiles; split the batch");
    a.total_tiles = uint32_t(total_tiles);
    const int grid = ar::step_grid(total_tiles);
    const int e = ar::launch_step(a, pl->dtype, pl->op, vec, nt, grid, stream);
    if (e != 0) return hip_fail(hipError_t(e), "step kernel launch");
    if (tm) tm->mark();
  }
  return AR_OK;
}

ar_status run_fused_lo(ar_plan* pl, void* const* bufs, int64_t batch, int64_t stride, hipStream_t stream,
                       int device, LaunchTimer* tm) {
  const ar::Schedule& s = pl->s;
  ar::FusedArgs a;
  std::memset(&a, 0, sizeof a);
  for (int32_t x = 0; x < s.P; ++x) a.user[x] = bufs[x];
  a.n = s.n;
  a.stride = stride;
  a.batch = batch;
  const int64_t cols = batch * s.n;
  const bool contiguous = (batch == 1 || stride == s.n);
  const int mode = contiguous ? 1 : 2;
  a.groups = cols;
  int64_t blocks = (a.groups + 255) / 256;
  blocks = std::min<int64_t>(std::max<int64_t>(blocks, 1), int64_t(1) << 22);
  const bool nt = mode == 1 && use_nt(pl->fused_nt_mode, int64_t(2) * s.P * cols * 4, kFusedNtThresholdBytes);
  a.lds = cap_lds(pl->fused_cap, device);
  if (tm) tm->mark();
  const int e = ar::launch_fused_lo(a, s.P, pl->dtype, pl->op, mode, nt, int(blocks), stream);
  if (e != 0) return hip_fail(hipError_t(e), "fused latency-optimal kernel launch");
  if (tm) tm->mark();
  return AR_OK;
}

ar_status run_fused_col(ar_plan* pl, void* const* bufs, int64_t batch, int64_t stride, hipStream_t stream,
                        int device, LaunchTimer* tm) {
  // one ColArgs layout for every column kernel; the XOR kernel reads the
  // first P entries of the rank table, the others a rotation of it
  const ar::Schedule& s = pl->s;
  ar::ColArgs a;
  std::memset(&a, 0, sizeof a);
  for (int32_t x = 0; x < 2 * s.P; ++x) a.user[x] = bufs[x % s.P];
  a.P = s.P;
  a.r = s.r;
  a.split = pl->fused_split ? 1 : 0;
  a.stride = stride;
  a.q = s.n / s.P;
  a.m = s.n % s.P;
  const int64_t max_len = a.q + (a.m ? 1 : 0);
  // +63: the tile grid of a block is shifted onto 256-byte boundaries
  const int64_t tiles = std::max<int64_t>(1, (max_len + 63 + 63) / 64);
  a.tiles = ar::make_fastdiv(uint32_t(std::min<int64_t>(tiles, INT32_MAX)));
  a.pdiv = ar::make_fastdiv(uint32_t(s.P));
  // Flat columns (the batch * n columns of all instances as one space, so
  // that small instances fill whole waves): latency-optimal plans, whose
  // trees are the same for every block, and sums with short blocks
  // (fused_flat) -- the rank-slot kernel, which rotates each lane's column by
  // its block, or the XOR group's kernel, whose sums do not see the block.
  const int64_t cols = batch * s.n;
  const bool flat_fits = cols < (int64_t(1) << 32) - 64;
  const bool flat_short = pl->fused_flat && flat_fits;
  if ((s.r == s.L && pl->fused_kind != kFusedRing && flat_fits) || flat_short) {
    a.flat = 1;
    a.flat_cols = uint32_t(cols);
    a.ndiv = ar::make_fastdiv(uint32_t(s.n));
    a.q1div = ar::make_fastdiv(uint32_t(a.q + 1));
    a.qdiv = ar::make_fastdiv(uint32_t(a.q > 0 ? a.q : 1));
    a.total_tiles = uint32_t((cols + 63) / 64);
  } else if (max_len >= 1 && batch < INT32_MAX &&
             (pl->packed_mode == 1 ? max_len <= int64_t(64)
                                   : pl->packed_mode < 0 && batch > 1 && max_len <= kPackMaxLen)) {
    // Short blocks: one block of 64 / max_len instances per wave tile.
    a.packed = 1;
    a.ipw = uint32_t(64 / max_len);
    a.batch = uint32_t(batch);
    a.lendiv = ar::make_fastdiv(uint32_t(max_len));
    const int64_t total = (batch + a.ipw - 1) / a.ipw * s.P;
    if (total >= (int64_t(1) << 31))
      return fail(AR_ERR_UNSUPPORTED, "the fused kernel would need 2^31 or more tiles; split the batch");
    a.total_tiles = uint32_t(total);
  } else {
    const int64_t total = batch * s.P * tiles;
    if (total >= (int64_t(1) << 31))
      return fail(AR_ERR_UNSUPPORTED, "the fused kernel would need 2^31 or more tiles; split the batch");
    a.total_tiles = uint32_t(total);
  }
  const bool nt = use_nt(pl->fused_nt_mode, int64_t(2) * s.P * s.n * batch * 4, kFusedNtThresholdBytes);
  const int grid = ar::step_grid(a.total_tiles);
  a.lds = cap_lds(pl->fused_cap, device);
  if (tm) tm->mark();
  int e;
  if (pl->fused_kind == kFusedXor) e = ar::launch_fused_xor(a, s.P, pl->dtype, pl->op, nt, grid, stream);
  else if (flat_short) e = ar::launch_fused_rot_any(a, s.P, pl->dtype, pl->op, pl->fused_kind == kFusedRing, grid, stream);
  else if (pl->fused_kind == kFusedRing) e = ar::launch_fused_ring(a, pl->dtype, pl->op, nt, grid, stream);
  else e = ar::launch_fused_col_any(a, s.P, pl->dtype, pl->op, nt, grid, stream);
  if (e != 0) return hip_fail(hipError_t(e), "column-fused kernel launch");
  if (tm) tm->mark();
  if (pl->fused_split) {
    // the tiled copy: nontemporal stores from kBcastStreamMinP ranks up, and
    // on flat columns at any P (P = 37: 11% faster, P = 48-128: 1-3%)
    const bool big = int64_t(s.P) * s.n * batch * 4 >= kFusedNtThresholdBytes;
    const bool bnt = pl->bcast_nt_mode == 1 ||
                     (pl->bcast_nt_mode < 0 && (s.P >= kBcastStreamMinP || flat_short) && big);
    ar::StreamArgs sa;
    const int64_t span = batch * s.n * 4;
    const bool want_stream =
        pl->bcast_stream_mode >= 1 || (pl->bcast_stream_mode < 0 && (a.flat || span >= kBcastStreamMinBytes));
    // chunks can straddle two blocks when a block or instance boundary is
    // not a multiple of the chunk
    const bool straddle = !a.flat && (s.n % s.P != 0 || (s.n / s.P) % ar::kStreamChunk != 0);
    bool regions;
    if (pl->bcast_stream_mode == 2 || pl->bcast_stream_mode == 3) regions = pl->bcast_stream_mode == 3;
    else if (a.flat) regions = span > kBcastFlatInterleaveMaxBytes;
    else if (!straddle) regions = s.P >= kBcastRegionMinP || span >= kBcastAlignedRegionMinBytes;
    else regions = s.P >= kBcastRegionMinP && span < kBcastInterleaveMinBytes;
    if (want_stream && stream_bcast_args(pl, bufs, batch, stride, a.flat != 0, regions, device, &sa)) {
      const uint32_t sgrid = (sa.chunks + sa.cdiv.d - 1) / sa.cdiv.d * sa.sdiv.d;
      // the destination-major copy: nontemporal at any P (launches of
      // kFusedNtThresholdBytes and more).  Alone, its cached stores were up
      // to 6% faster on some shapes (P = 64 at 16 MB per rank, flat columns),
      // but the pair then took 0.3-10% longer: the next reducing launch pays
      // for the cached lines (P = 32-128, 4-256 MB per rank, flat and block)
      const bool snt = pl->bcast_nt_mode == 1 || (pl->bcast_nt_mode < 0 && big);
      e = ar::launch_broadcast_stream(sa, snt, straddle, sgrid, stream);
    } else {
      a.lds = cap_lds(pl->bcast_cap, device);
      e = ar::launch_broadcast(a, pl->dtype, bnt, grid, stream);
    }
    if (e != 0) return hip_fail(hipError_t(e), "broadcast kernel launch");
    if (tm) tm->mark();
  }
  return AR_OK;
}

ar_status execute_impl(ar_plan* plan, void* const* rank_buffers, int64_t batch, int64_t instance_stride,
                       hipStream_t stream, LaunchTimer* tm, bool noalloc = false) {
  if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
  if (!rank_buffers) return fail(AR_ERR_INVALID_ARG, "rank_buffers is NULL");
  if (batch < 1) return fail(AR_ERR_INVALID_ARG, "batch must be >= 1");
  if (batch == 1 && instance_stride < plan->s.n) instance_stride = plan->s.n;
  if (instance_stride < plan->s.n) return fail(AR_ERR_INVALID_ARG, "instance_stride must be >= n");
  if (plan->s.n == 0) return AR_OK;  // nothing is read or written; the pointers may be NULL
  // one rank's extent, (batch - 1) * instance_stride + n elements, within
  // kMaxRankElems (n is, and instance_stride >= n >= 1 here)
  if (batch - 1 > (ar::kMaxRankElems - plan->s.n) / instance_stride)
    return fail(AR_ERR_INVALID_ARG, "a rank's extent, (batch - 1) * instance_stride + n, exceeds 2^46 elements");
  bool all16 = false;
  ar_status st = check_buffers(plan, rank_buffers, batch, instance_stride, &all16);
  if (st != AR_OK) return st;
  if (plan->s.P == 1) return AR_OK;  // nothing to combine
  int device = -1;
  hipError_t he = hipGetDevice(&device);
  if (he != hipSuccess) {
    (void)hipGetLastError();
    return fail(AR_ERR_NO_DEVICE, std::string("no usable GPU: ") + hipGetErrorString(he));
  }
  const bool fused = plan->path == AR_PATH_FUSED || (plan->path == AR_PATH_AUTO && plan->fused_ok);
  if (fused && plan->fused_kind != kFusedLo) {
    st = run_fused_col(plan, rank_buffers, batch, instance_stride, stream, device, tm);
  } else if (fused) {
    st = run_fused_lo(plan, rank_buffers, batch, instance_stride, stream, device, tm);
  } else {
    const bool vec = all16 && (batch == 1 || instance_stride % 4 == 0);
    st = run_stepwise(plan, rank_buffers, batch, instance_stride, vec, stream, device, tm, noalloc);
  }
  if (st == AR_OK) {
    plan->last_stream = stream;
    plan->ran = true;
  }
  return st;
}


// The plan as text (ar_plan_dump, AR_LOG=1): sizes, path choices and the
// step-wise launch tables.
std::string plan_text(const ar_plan* pl) {
  const ar::Schedule& s = pl->s;
  const bool xorg = s.group == ar::kGroupXor;
  std::string out;
  char line[256];
  auto add = [&out, &line](int len) {
    if (len > 0) out.append(line, size_t(std::min<int>(len, int(sizeof line) - 1)));
  };
  static const char* const kBuf[] = {"U", "X", "Y"};
  auto buf = [](int32_t b) { return b >= 0 && b <= 2 ? kBuf[b] : "-"; };
  add(std::snprintf(line, sizeof line, "ar_plan P=%d n=%lld dtype=%s op=%s group=%s schedule=%s k=%d L=%d r=%d w=%d\n",
                    s.P, (long long)s.n, pl->dtype == AR_INT32 ? "int32" : "float32", pl->op == AR_SUM ? "sum" : "max",
                    xorg ? "xor" : "cyclic", s.sched == ar::kSchedRing ? "ring" : "butterfly", s.k, s.L, s.r, s.w));
  add(std::snprintf(line, sizeof line,
                    "  steps: %d reduction + %d distribution; per rank and instance: %lld blocks pulled, %lld "
                    "combines; step-wise HBM %lld blocks, scratch %s\n",
                    s.rs_steps, s.ag_steps, (long long)s.blocks_pulled_per_rank, (long long)s.combines_per_rank,
                    (long long)s.hbm_blocks, s.uses_scratch ? "yes" : "no"));
  static const char* const kKind[] = {"none", "latency-optimal, registers", "cyclic butterfly columns", "XOR group columns",
                                      "Ring columns"};
  add(std::snprintf(line, sizeof line,
                    "  fused: %s; flat short blocks %s; split %s; caps %d/%d; path %s\n",
                    kKind[pl->fused_kind], pl->fused_flat ? "yes" : "no", pl->fused_split ? "yes" : "no", pl->fused_cap,
                    pl->bcast_cap,
                    pl->path == AR_PATH_STEPWISE ? "stepwise" : pl->path == AR_PATH_FUSED ? "fused" : "auto"));
  static const char* const kPhase[] = {"reduce", "distribute", "local copy"};
  static const char* const kRange[] = {"copy", "reduce", "reduce2"};
  for (size_t i = 0; i < s.launches.size(); ++i) {
    const ar::Launch& l = s.launches[i];
    add(std::snprintf(line, sizeof line, "  launch %zu (%s):", i, l.phase >= 0 && l.phase <= 2 ? kPhase[l.phase] : "?"));
    for (const ar::Range& r : l.ranges) {
      add(std::snprintf(line, sizeof line, xorg ? " [p %d..%d %s from x^%d: %s" : " [p %d..%d %s from x%+d: %s", r.p0,
                        r.p0 + r.count - 1, r.kind >= 0 && r.kind <= 2 ? kRange[r.kind] : "?", r.delta, buf(r.dst)));
      if (r.kind == ar::kCopy) add(std::snprintf(line, sizeof line, " = %s", buf(r.src)));
      else add(std::snprintf(line, sizeof line, " = %s (+) %s", buf(r.own), buf(r.src)));
      if (r.kind == ar::kReduce2)
        add(std::snprintf(line, sizeof line, ", %s = %s (+) %s", buf(r.dst2), buf(r.own2), buf(r.src)));
      out += ']';
    }
    out += '\n';
  }
  return out;
}
}  // namespace

namespace {

// Cost-model parameters for MI355X (gfx950), from the calibration sweeps
// (every k step by step and the fused path, P = 8, 37 and 127, messages of
// 2 KB to 4 GB, executes enqueued back to back from Python): the fitted
// per-launch cost was 4.7-7.2 us and the step launches' effective bandwidth
// 7-11 TB/s of their algorithmic bytes (the smaller steps stay in the 256 MB
// Infinity Cache).  Of the values tried, these chose a step count within
// 6.3% of the fastest measured at every size (1% on average); the fused path
// was faster than every step count at every size, as these values price it.
constexpr ar_model_params kDefaultModel = {5.0e-6, 7.0e12, 5.0e-6, 6.0e12};

bool model_params_ok(const ar_model_params& mp) {
  return mp.step_alpha >= 0 && mp.fused_alpha >= 0 && mp.step_bytes_per_s > 0 && mp.fused_bytes_per_s > 0 &&
         std::isfinite(mp.step_alpha) && std::isfinite(mp.fused_alpha) && std::isfinite(mp.step_bytes_per_s) &&
         std::isfinite(mp.fused_bytes_per_s);
}

// Sec. 2's model on one GPU: every launch costs alpha, and its HBM bytes
// cost 1 / bandwidth each (P ranks share the device).
double model_seconds(const ar_plan* pl, const ar_model_params& mp, int64_t batch, int32_t path) {
  const ar::Schedule& s = pl->s;
  if (s.P < 2 || s.n == 0) return 0.0;
  if (path == AR_PATH_FUSED) {
    const double launches = pl->fused_split ? 2.0 : 1.0;
    const double bytes = double(int64_t(2) * s.P + (pl->fused_split ? 1 : 0)) * double(s.n) * 4.0 * double(batch);
    return launches * mp.fused_alpha + bytes / mp.fused_bytes_per_s;
  }
  const double bytes = double(s.hbm_blocks) * double(s.n) * 4.0 * double(batch);
  return double(s.launches.size()) * mp.step_alpha + bytes / mp.step_bytes_per_s;
}

// Plan creation proper (ar_plan_create_ex without AR_K_AUTO); `log` lets
// AR_LOG=1 print the plan (not the candidates the automatic choice prices).
ar_status create_plan(int32_t P, int64_t n, ar_dtype dtype, ar_op op, int32_t k_steps, ar_group group,
                      ar_schedule schedule, bool log, ar_plan** out_plan) {
  if (!out_plan) return fail(AR_ERR_INVALID_ARG, "out_plan is NULL");
  *out_plan = nullptr;
  if (int(dtype) != AR_INT32 && int(dtype) != AR_FLOAT32) return fail(AR_ERR_UNSUPPORTED, "dtype must be int32 or float32");
  if (int(op) != AR_SUM && int(op) != AR_MAX) return fail(AR_ERR_UNSUPPORTED, "op must be sum or max");
  if (P > ar::kMaxP) return fail(AR_ERR_UNSUPPORTED, "P above the compiled maximum of 128 ranks");
  if (int(group) != AR_GROUP_CYCLIC && int(group) != AR_GROUP_XOR) return fail(AR_ERR_INVALID_ARG, "unknown group");
  if (int(schedule) != AR_SCHEDULE_BUTTERFLY && int(schedule) != AR_SCHEDULE_RING)
    return fail(AR_ERR_INVALID_ARG, "unknown schedule");
  ar_plan* pl = new (std::nothrow) ar_plan;
  if (!pl) return fail(AR_ERR_OUT_OF_MEMORY, "plan allocation");
  const std::string err = ar::build_schedule_ex(P, n, k_steps, int32_t(group), int32_t(schedule), &pl->s);
  if (!err.empty()) {
    delete pl;
    return fail(err.rfind("internal", 0) == 0 ? AR_ERR_INTERNAL : AR_ERR_INVALID_ARG, err);
  }
  pl->dtype = int32_t(dtype);
  pl->op = int32_t(op);
  auto env_mode = [](const char* name) {
    const char* e = std::getenv(name);
    return e == nullptr ? -1 : (e[0] == '1') ? 1 : (e[0] == '0') ? 0 : -1;
  };
  pl->nt_mode = env_mode("AR_STEP_NT");
  pl->fused_nt_mode = env_mode("AR_FUSED_NT");
  pl->split_mode = env_mode("AR_FUSED_SPLIT");
  pl->bcast_nt_mode = env_mode("AR_BCAST_NT");
  {
    // 0: tiled; 1: destination-major, chunk order by size; 2 / 3: destination-major with
    // interleaved chunks / XCD regions
    const char* e = std::getenv("AR_BCAST_STREAM");
    pl->bcast_stream_mode = e != nullptr && e[0] >= '0' && e[0] <= '3' && e[1] == 0 ? int32_t(e[0] - '0') : -1;
  }
  pl->packed_mode = env_mode("AR_FUSED_PACKED");
  pl->rotate_mode = env_mode("AR_FUSED_ROTATE");
  pl->merge_mode = env_mode("AR_STEP_MERGE");
  if (pl->s.P < 2) pl->fused_kind = kFusedNone;
  else if (pl->s.sched == ar::kSchedRing) pl->fused_kind = kFusedRing;
  else if (pl->s.group == ar::kGroupXor) pl->fused_kind = kFusedXor;
  else if (pl->s.P <= ar::kFusedMaxP && pl->s.r == pl->s.L) pl->fused_kind = kFusedLo;
  else pl->fused_kind = kFusedCol;
  pl->fused_ok = pl->fused_kind != kFusedNone;
  // one result for every rank: the Ring, and r = 0 outside the flat LO kernel
  const bool one_result = pl->fused_kind == kFusedRing ||
                          ((pl->fused_kind == kFusedCol || pl->fused_kind == kFusedXor) && pl->s.r == 0);
  {
    const int64_t max_len = pl->s.P > 0 ? pl->s.n / pl->s.P + (pl->s.n % pl->s.P ? 1 : 0) : 0;
    const bool kind = pl->fused_kind == kFusedRing || pl->fused_kind == kFusedXor ||
                      (pl->fused_kind == kFusedCol && pl->s.r < pl->s.L);
    // max: the rank-slot kernel's bandwidth-optimal fold and Ring, its
    // shifted plans at P = kRotMaxShiftedMinP-kRotMaxShiftedMaxP (elsewhere
    // they keep block or packed tiles, saving their instantiations), and the
    // XOR group, whose flat kernel then takes each lane's block
    const bool max_mid_p = pl->s.P >= ar::kRotMaxShiftedMinP && pl->s.P <= ar::kRotMaxShiftedMaxP;
    const bool op_ok = pl->op == AR_SUM || pl->fused_kind == kFusedRing || pl->fused_kind == kFusedXor ||
                       (pl->fused_kind == kFusedCol && (pl->s.r == 0 || max_mid_p));
    const bool shifted = pl->fused_kind == kFusedCol && pl->s.r > 0;
    const bool small_p = pl->s.P >= kRotShiftedSmallMinP && pl->s.P <= kRotShiftedSmallMaxP &&
                         pl->s.n * 4 <= kRotShiftedSmallMaxBytes;
    const bool rot_shifted =
        shifted && ((pl->op == AR_SUM && pl->s.P >= kRotShiftedMinP && pl->s.P % 2 == 1) ||
                    (small_p && (pl->op == AR_SUM || max_mid_p)));
    const bool rot_one = (pl->fused_kind == kFusedRing || (pl->fused_kind == kFusedCol && pl->s.r == 0)) &&
                         pl->s.P >= kRotOneMinP && pl->s.n * 4 < kRotOneMaxBytes;
    const bool xor_long = pl->fused_kind == kFusedXor && pl->s.r < pl->s.L;
    pl->fused_flat =
        kind && op_ok &&
        (pl->rotate_mode == 1 ||
         (pl->rotate_mode < 0 && (max_len <= kPackMaxLen || rot_shifted || rot_one || xor_long)));
  }
  const bool rank_slots = pl->fused_flat && pl->fused_kind != kFusedXor;
  const int32_t split_min =
      rank_slots ? kFlatSplitMinP : (pl->s.n * 4 >= kSplitMidMinBytes ? kSplitMidMinP : kSplitMinP);
  pl->fused_split = one_result && (pl->split_mode == 1 || (pl->split_mode < 0 && pl->s.P >= split_min));
  {
    const int32_t P = pl->s.P;
    if (pl->fused_split) pl->fused_cap = (rank_slots && P < kSplitMinP) ? 4 : 6;
    else if (pl->fused_flat) pl->fused_cap = P <= 6 ? 0 : P <= 8 ? 6 : P <= 16 ? 4 : P < 64 ? 2 : 0;
    else if (pl->fused_kind == kFusedLo) pl->fused_cap = lo_cap(P);
    else if (P <= 8) pl->fused_cap = P <= 6 ? 0 : 6;  // few rank rows per wave: more waves resident
    else if (pl->fused_kind == kFusedRing) pl->fused_cap = 4;
    else if (pl->s.r == 0) pl->fused_cap = P <= 32 ? 4 : 3;
    else pl->fused_cap = P >= 64 ? 0 : 3;
    pl->bcast_cap = P >= kBcastStreamMinP ? 1 : 2;
    // AR_FUSED_CAP = N caps both launches, "N,M" the fused one and the broadcast
    // (values clamped to [0, 64]; 0 means no cap)
    auto cap_of = [](const char* str) { return int32_t(std::min(std::strtol(str, nullptr, 10), 64L)); };
    const char* ce = std::getenv("AR_FUSED_CAP");
    if (ce != nullptr && ce[0] >= '0' && ce[0] <= '9') {
      pl->fused_cap = pl->bcast_cap = cap_of(ce);
      const char* comma = std::strchr(ce, ',');
      if (comma != nullptr && comma[1] >= '0' && comma[1] <= '9') pl->bcast_cap = cap_of(comma + 1);
    }
  }
  if (log && env_mode("AR_LOG") == 1) std::fputs(plan_text(pl).c_str(), stderr);
  *out_plan = pl;
  g_err.clear();
  return AR_OK;
}

}  // namespace

extern "C" {

ar_status ar_plan_create_ex(int32_t P, int64_t n, ar_dtype dtype, ar_op op, int32_t k_steps, ar_group group,
                            ar_schedule schedule, ar_plan** out_plan) {
  if (k_steps == AR_K_AUTO) {
    if (!out_plan) return fail(AR_ERR_INVALID_ARG, "out_plan is NULL");
    *out_plan = nullptr;
    if (int(schedule) != AR_SCHEDULE_BUTTERFLY)
      return fail(AR_ERR_INVALID_ARG, "AR_K_AUTO chooses among the butterfly schedules only");
    return ar_plan_create_auto(P, n, dtype, op, group, 1, AR_PATH_AUTO, nullptr, out_plan);
  }
  return create_plan(P, n, dtype, op, k_steps, group, schedule, true, out_plan);
}

ar_status ar_plan_create(int32_t P, int64_t n, ar_dtype dtype, ar_op op, int32_t k_steps, ar_plan** out_plan) {
  return ar_plan_create_ex(P, n, dtype, op, k_steps, AR_GROUP_CYCLIC, AR_SCHEDULE_BUTTERFLY, out_plan);
}

ar_status ar_plan_set_path(ar_plan* plan, ar_path path) {
  if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
  if (path != AR_PATH_AUTO && path != AR_PATH_STEPWISE && path != AR_PATH_FUSED)
    return fail(AR_ERR_INVALID_ARG, "unknown path");
  if (path == AR_PATH_FUSED && !plan->fused_ok)
    return fail(AR_ERR_UNSUPPORTED, "a single rank has nothing to fuse");
  plan->path = path;
  return AR_OK;
}

ar_status ar_execute_batched(ar_plan* plan, void* const* rank_buffers, int64_t batch, int64_t instance_stride,
                             hipStream_t stream) {
  return execute_impl(plan, rank_buffers, batch, instance_stride, stream, nullptr);
}

ar_status ar_execute_noalloc(ar_plan* plan, void* const* rank_buffers, int64_t batch, int64_t instance_stride,
                             hipStream_t stream) {
  return execute_impl(plan, rank_buffers, batch, instance_stride, stream, nullptr, true);
}

ar_status ar_execute(ar_plan* plan, void* const* rank_buffers, hipStream_t stream) {
  return ar_execute_batched(plan, rank_buffers, 1, plan ? plan->s.n : 0, stream);
}

ar_status ar_execute_timed(ar_plan* plan, void* const* rank_buffers, int64_t batch, int64_t instance_stride,
                           hipStream_t stream, float* launch_ms, int32_t cap, int32_t* n_launches) {
  if (!n_launches) return fail(AR_ERR_INVALID_ARG, "n_launches is NULL");
  if (cap < 0 || (cap > 0 && !launch_ms)) return fail(AR_ERR_INVALID_ARG, "launch_ms is NULL or cap < 0");
  *n_launches = 0;
  LaunchTimer tm;
  tm.stream = stream;
  ar_status st = execute_impl(plan, rank_buffers, batch, instance_stride, stream, &tm);
  if (st != AR_OK) return st;
  if (tm.err != hipSuccess) return hip_fail(tm.err, "timing event");
  if (tm.ev.empty()) return AR_OK;  // nothing was launched (n = 0 or P = 1)
  hipError_t e = hipEventSynchronize(tm.ev.back());
  if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
  const int32_t n = int32_t(tm.ev.size()) - 1;
  for (int32_t i = 0; i < n && i < cap; ++i) {
    float ms = 0.0f;
    e = hipEventElapsedTime(&ms, tm.ev[size_t(i)], tm.ev[size_t(i) + 1]);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    launch_ms[i] = ms;
  }
  *n_launches = n;
  return AR_OK;
}

ar_status ar_plan_stats(const ar_plan* plan, ar_stats* out) {
  if (!plan || !out) return fail(AR_ERR_INVALID_ARG, "NULL argument");
  const ar::Schedule& s = plan->s;
  std::memset(out, 0, sizeof *out);
  out->P = s.P;
  out->L = s.L;
  out->k = s.k;
  out->r = s.r;
  out->w = s.w;
  out->rs_steps = s.rs_steps;
  out->ag_steps = s.ag_steps;
  out->launches = int32_t(s.launches.size());
  out->fused_ok = plan->fused_ok ? 1 : 0;
  out->n = s.n;
  out->elem_bytes = 4;
  out->blocks_pulled_per_rank = s.blocks_pulled_per_rank;
  // bytes: rank x pulls block (x - p) for every pulled placement p
  int64_t mn = INT64_MAX, mx = 0, total = 0;
  for (int32_t x = 0; x < s.P; ++x) {
    int64_t bytes = 0;
    for (const ar::Launch& l : s.launches) {
      std::vector<char> seen(size_t(3) * s.P, 0);
      for (const ar::Range& rg : l.ranges) {
        if (rg.delta == 0) continue;
        for (int32_t j = 0; j < rg.count; ++j) {
          const int32_t p = (rg.p0 + j) % s.P;
          char& sn = seen[size_t(rg.src) * s.P + p];
          if (sn) continue;
          sn = 1;
          const int32_t b = ar::group_block(s.group, x, p, s.P);
          bytes += ar::block_len(s.n, s.P, b) * 4;
        }
      }
    }
    mn = std::min(mn, bytes);
    mx = std::max(mx, bytes);
    total += bytes;
  }
  out->bytes_pulled_per_rank_min = s.P ? mn : 0;
  out->bytes_pulled_per_rank_max = mx;
  out->bytes_pulled_total = total;
  out->combines_per_rank = s.combines_per_rank;
  out->hbm_bytes_stepwise = s.hbm_blocks * s.n * 4;
  out->hbm_bytes_fused = s.P > 1 ? (int64_t(2) * s.P + (plan->fused_split ? 1 : 0)) * s.n * 4 : 0;
  out->fused_launches = s.P > 1 ? (plan->fused_split ? 2 : 1) : 0;
  out->fused_flat = s.P > 1 && plan->fused_flat ? 1 : 0;
  out->workspace_bytes = s.uses_scratch ? int64_t(2) * s.P * round_up(s.n, 64) * 4 : 0;
  out->group = s.group;
  out->schedule = s.sched;
  out->exec_path = s.P < 2 ? 0 : (plan->path == AR_PATH_FUSED || (plan->path == AR_PATH_AUTO && plan->fused_ok))
                                     ? AR_PATH_FUSED
                                     : AR_PATH_STEPWISE;
  out->hbm_bytes_algorithmic = out->hbm_bytes_stepwise;
  {
    // the default choice for one instance (ar.h): flat columns, and blocks
    // of at least kStreamChunk elements in rank buffers of at least
    // kBcastStreamMinBytes
    const bool flat = plan->fused_flat;
    const bool allowed = flat || s.n / std::max<int32_t>(s.P, 1) >= int64_t(ar::kStreamChunk);
    const bool by_size = flat || s.n * 4 >= kBcastStreamMinBytes;
    out->fused_bcast_stream =
        s.P > 1 && plan->fused_split && allowed && (plan->bcast_stream_mode >= 1 || (plan->bcast_stream_mode < 0 && by_size))
            ? 1
            : 0;
  }
  return AR_OK;
}

ar_status ar_plan_dump(const ar_plan* plan, char* buf, int64_t cap, int64_t* len) {
  if (!plan || !len) return fail(AR_ERR_INVALID_ARG, "NULL argument");
  if (cap < 0 || (cap > 0 && !buf)) return fail(AR_ERR_INVALID_ARG, "buf is NULL or cap < 0");
  const std::string t = plan_text(plan);
  *len = int64_t(t.size());
  if (cap > 0) {
    const size_t k = std::min<size_t>(t.size(), size_t(cap - 1));
    std::memcpy(buf, t.data(), k);
    buf[k] = 0;
  }
  return AR_OK;
}

ar_status ar_plan_num_launches(const ar_plan* plan, int32_t* out) {
  if (!plan || !out) return fail(AR_ERR_INVALID_ARG, "NULL argument");
  *out = int32_t(plan->s.launches.size());
  return AR_OK;
}

ar_status ar_plan_launch(const ar_plan* plan, int32_t i, ar_launch_desc* desc, ar_range_desc* ranges, int32_t cap) {
  if (!plan || !desc) return fail(AR_ERR_INVALID_ARG, "NULL argument");
  if (i < 0 || i >= int32_t(plan->s.launches.size())) return fail(AR_ERR_INVALID_ARG, "launch index out of range");
  const ar::Launch& l = plan->s.launches[i];
  desc->phase = l.phase;
  desc->n_ranges = int32_t(l.ranges.size());
  if (ranges) {
    for (int32_t j = 0; j < desc->n_ranges && j < cap; ++j) {
      const ar::Range& r = l.ranges[j];
      ranges[j] = ar_range_desc{r.p0, r.count, r.kind, r.delta, r.dst, r.own, r.dst2, r.own2, r.src};
    }
  }
  return AR_OK;
}

ar_status ar_model_time(int32_t P, double m_bytes, int32_t k_steps, double alpha, double beta, double gamma,
                        double* tau_seconds) {
  if (!tau_seconds) return fail(AR_ERR_INVALID_ARG, "tau_seconds is NULL");
  if (P < 1 || P > ar::kMaxP) return fail(AR_ERR_INVALID_ARG, "P must be in [1, 128]");
  if (!(m_bytes >= 0) || !(alpha >= 0) || !(beta >= 0) || !(gamma >= 0))
    return fail(AR_ERR_INVALID_ARG, "m, alpha, beta and gamma must be >= 0");
  int32_t L = 0;
  while ((1 << L) < P) ++L;
  if (k_steps < L || k_steps > 2 * L) return fail(AR_ERR_INVALID_ARG, "k_steps outside [L, 2L]");
  const int32_t r = 2 * L - k_steps;
  const double u = m_bytes / P;
  double t;
  if (P == 1) {
    t = 0.0;
  } else if (r == 0) {  // Sec. 7
    t = 2.0 * L * alpha + 2.0 * (P - 1) * u * beta + double(P - 1) * u * gamma;
  } else if (r == L) {  // Sec. 9
    t = double(L) * alpha + double(P) * L * u * beta + double(P) * (2 * L - 2) * u * gamma;
  } else {              // Sec. 8
    const double x = double((int64_t(1) << r) - 1);
    t = double(2 * L - r) * alpha + (2.0 * (P - 1) + x * (L - 1)) * u * beta + ((P - 1) + x * (2 * L - 2)) * u * gamma;
  }
  *tau_seconds = t;
  return AR_OK;
}

ar_status ar_model_best_k(int32_t P, double m_bytes, double alpha, double beta, double gamma, int32_t* k_steps,
                          double* r_closed_form) {
  if (!k_steps) return fail(AR_ERR_INVALID_ARG, "k_steps is NULL");
  if (P < 1 || P > ar::kMaxP) return fail(AR_ERR_INVALID_ARG, "P must be in [1, 128]");
  int32_t L = 0;
  while ((1 << L) < P) ++L;
  double best = 0;
  int32_t best_k = -1;
  for (int32_t k = L; k <= 2 * L; ++k) {
    double t = 0;
    const ar_status st = ar_model_time(P, m_bytes, k, alpha, beta, gamma, &t);
    if (st != AR_OK) return st;
    if (best_k < 0 || t < best) {
      best = t;
      best_k = k;
    }
  }
  *k_steps = best_k;
  if (r_closed_form) {
    // Sec. 8: r* = log2(alpha / (m (beta + 2 gamma))) + log2(P / ((log2 P - 1) ln 2))
    const double lp = std::log2(double(P));
    const double den = m_bytes * (beta + 2 * gamma);
    *r_closed_form = (P > 2 && den > 0 && alpha > 0)
                         ? std::log2(alpha / den) + std::log2(double(P) / ((lp - 1.0) * std::log(2.0)))
                         : std::nan("");
  }
  return AR_OK;
}

ar_status ar_plan_model_time(const ar_plan* plan, double alpha, double beta, double gamma, double* tau_seconds) {
  if (!plan || !tau_seconds) return fail(AR_ERR_INVALID_ARG, "NULL argument");
  if (!(alpha >= 0) || !(beta >= 0) || !(gamma >= 0)) return fail(AR_ERR_INVALID_ARG, "negative model parameter");
  const ar::Schedule& s = plan->s;
  const double u = double(s.n) * 4 / s.P;  // bytes per (average) block
  *tau_seconds = double(s.k) * alpha + double(s.blocks_pulled_per_rank) * u * beta +
                 double(s.combines_per_rank) * u * gamma;
  return AR_OK;
}

ar_status ar_model_default_params(ar_model_params* out) {
  if (!out) return fail(AR_ERR_INVALID_ARG, "out is NULL");
  *out = kDefaultModel;
  return AR_OK;
}

ar_status ar_plan_model_seconds(const ar_plan* plan, const ar_model_params* params, int64_t batch, ar_path path,
                                double* seconds) {
  if (!plan || !seconds) return fail(AR_ERR_INVALID_ARG, "NULL argument");
  if (batch < 1) return fail(AR_ERR_INVALID_ARG, "batch must be >= 1");
  const ar_model_params& mp = params ? *params : kDefaultModel;
  if (!model_params_ok(mp)) return fail(AR_ERR_INVALID_ARG, "model alphas must be >= 0 and bandwidths > 0");
  if (path != AR_PATH_AUTO && path != AR_PATH_STEPWISE && path != AR_PATH_FUSED)
    return fail(AR_ERR_INVALID_ARG, "unknown path");
  if (path == AR_PATH_AUTO)
    path = plan->path == AR_PATH_FUSED || (plan->path == AR_PATH_AUTO && plan->fused_ok) ? AR_PATH_FUSED
                                                                                         : AR_PATH_STEPWISE;
  if (path == AR_PATH_FUSED && !plan->fused_ok) return fail(AR_ERR_UNSUPPORTED, "the plan cannot run fused");
  *seconds = model_seconds(plan, mp, batch, path);
  return AR_OK;
}

ar_status ar_plan_create_auto(int32_t P, int64_t n, ar_dtype dtype, ar_op op, ar_group group, int64_t batch,
                              ar_path path, const ar_model_params* params, ar_plan** out_plan) {
  if (!out_plan) return fail(AR_ERR_INVALID_ARG, "out_plan is NULL");
  *out_plan = nullptr;
  if (batch < 1) return fail(AR_ERR_INVALID_ARG, "batch must be >= 1");
  if (path != AR_PATH_AUTO && path != AR_PATH_STEPWISE && path != AR_PATH_FUSED)
    return fail(AR_ERR_INVALID_ARG, "unknown path");
  const ar_model_params& mp = params ? *params : kDefaultModel;
  if (!model_params_ok(mp)) return fail(AR_ERR_INVALID_ARG, "model alphas must be >= 0 and bandwidths > 0");
  if (P > ar::kMaxP) return fail(AR_ERR_UNSUPPORTED, "P above the compiled maximum of 128 ranks");
  if (P < 1) return fail(AR_ERR_INVALID_ARG, "P must be in [1, 128]");
  int32_t L = 0;
  while ((1 << L) < P) ++L;
  // Sec. 8: the number of steps that the model prices cheapest on the
  // step-by-step schedule; the smallest k on a tie
  ar_plan* best = nullptr;
  double best_t = 0;
  for (int32_t k = L; k <= 2 * L; ++k) {
    ar_plan* p = nullptr;
    const ar_status st = create_plan(P, n, dtype, op, k, group, AR_SCHEDULE_BUTTERFLY, false, &p);
    if (st != AR_OK) {
      ar_plan_destroy(best);
      return st;
    }
    const double t = model_seconds(p, mp, batch, AR_PATH_STEPWISE);
    if (!best || t < best_t) {
      ar_plan_destroy(best);
      best = p;
      best_t = t;
    } else {
      ar_plan_destroy(p);
    }
  }
  ar_path chosen = path;
  if (path == AR_PATH_FUSED && !best->fused_ok) {
    ar_plan_destroy(best);
    return fail(AR_ERR_UNSUPPORTED, "a single rank has nothing to fuse");
  }
  if (path == AR_PATH_AUTO)
    chosen = best->fused_ok && model_seconds(best, mp, batch, AR_PATH_FUSED) < best_t ? AR_PATH_FUSED
                                                                                     : AR_PATH_STEPWISE;
  best->path = chosen;
  auto env_on = [](const char* name) {
    const char* e = std::getenv(name);
    return e != nullptr && e[0] == '1';
  };
  if (env_on("AR_LOG")) std::fputs(plan_text(best).c_str(), stderr);
  *out_plan = best;
  g_err.clear();
  return AR_OK;
}

void ar_plan_destroy(ar_plan* plan) {
  if (!plan) return;
  if (plan->scratch) plan->retired.push_back({plan->scratch, plan->scratch_device});
  if (!plan->retired.empty()) {
    // hipFree waits for the device to finish the work that still uses it
    int cur = 0;
    (void)hipGetDevice(&cur);
    for (const auto& r : plan->retired) {
      (void)hipSetDevice(r.second);
      (void)hipFree(r.first);
    }
    (void)hipSetDevice(cur);
  }
  delete plan;
}

const char* ar_status_string(ar_status s) {
  switch (s) {
    case AR_OK: return "ok";
    case AR_ERR_INVALID_ARG: return "invalid argument";
    case AR_ERR_UNSUPPORTED: return "unsupported";
    case AR_ERR_ALIAS: return "rank buffers overlap";
    case AR_ERR_OUT_OF_MEMORY: return "out of device memory";
    case AR_ERR_HIP: return "HIP runtime error";
    case AR_ERR_NO_DEVICE: return "no usable GPU";
    case AR_ERR_INTERNAL: return "internal consistency check failed";
  }
  return "unknown status";
}

const char* ar_last_error_message(void) { return g_err.c_str(); }

const char* ar_last_error(void) { return g_err.c_str(); }

}  // extern "C"
