// ar_internal.hpp -- types shared by the host plan generator, the C ABI and
// the HIP kernels of libar.so.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace ar {

constexpr int kMaxP = 128;       // largest supported number of ranks
constexpr int kMaxRanges = 8;    // placement ranges per launch
// Largest extent of one rank's buffer, in elements (2^46: 256 TiB of 4-byte
// elements, far above any device's memory), so that every size derived from
// it -- bytes, tiles, products with P -- fits in 64-bit arithmetic.
constexpr int64_t kMaxRankElems = int64_t(1) << 46;
constexpr int kFusedMaxP = 16;   // largest P of the register-resident fused kernel
// P range in which the rank-slot kernel also takes shifted max plans (the
// library instantiates those only there)
constexpr int kRotMaxShiftedMinP = 24, kRotMaxShiftedMaxP = 48;
// Size of the device-resident scratch of ar_execute_noalloc (noalloc.hip):
// the X and Y buffers of a step-wise plan with r > 0 take 2 * P rank
// regions of the call's extent rounded up to 64 elements.
constexpr int64_t kNoAllocScratchBytes = int64_t(64) << 20;

enum Buf : int32_t { kBufNone = -1, kBufU = 0, kBufX = 1, kBufY = 2 };
enum Kind : int32_t { kCopy = 0, kReduce = 1, kReduce2 = 2 };
enum Phase : int32_t { kPhaseReduce = 0, kPhaseDistribute = 1, kPhaseLocal = 2 };
// The group T_P (Sec. 5): cyclic, t_k(x) = x + k mod P, or the group of
// Table 1b for power-of-two P, t_k(x) = x XOR k.  Schedules: the butterfly
// family of Secs. 7-9 (any k in [L, 2L]) or the Ring of Sec. 6.
enum Group : int32_t { kGroupCyclic = 0, kGroupXor = 1 };
enum Sched : int32_t { kSchedButterfly = 0, kSchedRing = 1 };

// Block held at placement p by rank x (h = identity), and the rank a step
// with "delta" pulls from: x - p and x + delta mod P in the cyclic group,
// x XOR p and x XOR delta in the XOR group.
inline int32_t group_block(int32_t group, int32_t x, int32_t p, int32_t P) {
  if (group == kGroupXor) return x ^ p;
  const int32_t b = (x - p) % P;
  return b < 0 ? b + P : b;
}
inline int32_t group_peer(int32_t group, int32_t x, int32_t delta, int32_t P) {
  if (group == kGroupXor) return x ^ delta;
  const int32_t y = (x + delta) % P;
  return y < 0 ? y + P : y;
}

// One range of placements worked on by every rank in a launch.  delta names
// the peer (group_peer); the peer's copy of the same block is its placement
// p + delta (cyclic) or p XOR delta (XOR group).
struct Range {
  int32_t p0, count, kind, delta;
  int32_t dst, own, dst2, own2, src;
};

struct Launch {
  int32_t phase;
  std::vector<Range> ranges;
};

// The schedule and its sizes; built on the host (plan.cpp).
struct Schedule {
  int32_t P = 1, L = 0, k = 0, r = 0, w = 1;
  int32_t group = kGroupCyclic, sched = kSchedButterfly;
  int64_t n = 0;
  std::vector<int32_t> N, f, c;  // N_i, floor(N_i/2), ceil(N_i/2)
  std::vector<Launch> launches;
  int32_t rs_steps = 0, ag_steps = 0;
  bool uses_scratch = false;
  // sizes per instance
  int64_t blocks_pulled_per_rank = 0;
  int64_t combines_per_rank = 0;
  int64_t hbm_blocks = 0;  // block reads + writes per rank, STEPWISE path
};

// Builds the schedule; returns an empty string or the reason it failed.
std::string build_schedule(int32_t P, int64_t n, int32_t k, Schedule* out);
std::string build_schedule_ex(int32_t P, int64_t n, int32_t k, int32_t group, int32_t sched, Schedule* out);

// Verifies that no launch of `s` lets one work item write a location that a
// different work item reads or writes.  Returns "" or a description.
std::string check_hazards(const Schedule& s);

// Balanced partition: block b of n elements over P blocks.
inline int64_t block_off(int64_t n, int32_t P, int32_t b) {
  const int64_t q = n / P, m = n % P;
  return b * q + (b < m ? b : m);
}
inline int64_t block_len(int64_t n, int32_t P, int32_t b) {
  const int64_t q = n / P, m = n % P;
  return q + (b < m ? 1 : 0);
}

// Division of 32-bit numbers by a divisor fixed for a launch: a multiply-high
// and two shifts instead of a division sequence (unsigned division by
// invariant integers, Granlund & Montgomery 1994, "round-up" variant).
struct FastDiv {
  uint32_t d, m, l;  // divisor, magic multiplier, ceil(log2 d)
};

inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f{d, 0, 0};
  while ((uint64_t(1) << f.l) < d) ++f.l;
  f.m = uint32_t(((uint64_t(1) << 32) * ((uint64_t(1) << f.l) - d)) / d + 1);
  return f;
}

// Host reference of the device quotient (used by the tests).
inline uint32_t fastdiv_host(uint32_t n, const FastDiv& f) {
  if (f.l == 0) return n;
  const uint32_t t = uint32_t((uint64_t(n) * f.m) >> 32);
  return (t + ((n - t) >> 1)) >> (f.l - 1);
}

// ----- device launch interface (kernels.hip) -----

struct DevRange {
  int32_t p0, count, kind, delta;
  int32_t dst, own, dst2, own2, src;
  int32_t first;  // index of the range's first op among the launch's ops
};

struct StepArgs {
  void* user[kMaxP];        // rank buffers
  char* scratch[2];         // X and Y: rank y's region at scratch[i] + y * scratch_rank_stride elements
  int64_t scratch_rank_stride;
  int64_t n, stride;
  int64_t q, m;             // n / P, n % P
  uint32_t total_tiles;     // P * total_ops * batch * tiles_per_seg (< 2^31)
  FastDiv tps, batch, ops;  // tiles per segment, instances, ops per rank
  int32_t P, n_ranges;
  int32_t group;            // kGroupCyclic or kGroupXor
  DevRange ranges[kMaxRanges];
  // Merged runs (step_merged_kernel): the placements p0 .. p0+count-1 of a
  // range touch one run of consecutive blocks of rank x (cyclically), with
  // one peer and one set of buffers, so the range is streamed as one flat
  // space per rank: run_len[i] elements per instance (the whole row when
  // the range covers every placement, else count * ceil(n / P) -- a rank's
  // run is at most that long), batch * run_len[i] columns in all, tiles of
  // 256 columns.  Range i's tiles start at tile_first[i], P * tiles[i] of
  // them (rank-major).
  FastDiv run_len[kMaxRanges], tiles[kMaxRanges];
  uint32_t run_cols[kMaxRanges], tile_first[kMaxRanges];
};

// lds: dynamic LDS each workgroup reserves without using it, so that fewer
// workgroups are resident per CU (0: no cap); read by the launchers.
struct FusedArgs {
  void* user[kMaxP];
  int64_t n, stride, batch;
  int64_t groups;           // column groups (16-byte mode) or columns (other modes)
  uint32_t lds;
};

// Column kernels: wave tile t -> (instance, block, 64 columns of the block).
// The rank table is stored twice over (user[x] == user[x + P]) so that the
// ranks b, b+1, ..., b+P-1 of a rotation are consecutive entries.
struct ColArgs {
  void* user[2 * kMaxP];
  int64_t stride, q, m;     // instance stride, n / P, n % P
  uint32_t total_tiles;     // batch * P * tiles (< 2^31)
  FastDiv tiles, pdiv;      // column tiles per block, P
  int32_t P, r;             // r: distribution steps removed (kept shifts w = min(2^r, P))
  int32_t split;            // 1: store the block's result to its root rank only (a broadcast follows)
  uint32_t lds;             // as in FusedArgs
  // Latency-optimal plans (r = L): the tree of every rank is the same for
  // every block, so the kernels may tile the batch * n columns as one flat
  // space (64 per wave, no block index): flat = 1, flat_cols = batch * n
  // (< 2^32 - 64), ndiv = n.
  int32_t flat;
  uint32_t flat_cols;
  FastDiv ndiv;
  // Short blocks (every other plan): with packed = 1 a wave tile covers the
  // same block of ipw instances, lane = j * maxlen + c for column c of
  // instance j of the tile's group; lendiv = maxlen (the longest block),
  // ipw = 64 / maxlen, batch = the number of instances.  Otherwise a tile
  // covers 64 columns of one block of one instance.
  int32_t packed;
  uint32_t ipw, batch;
  FastDiv lendiv;
  // Rank-slot kernel of the cyclic butterfly plans (flat columns, block of
  // each lane from its index i in the instance): the first m blocks hold
  // q + 1 elements (q1div = q + 1), the others q (qdiv = max(q, 1)).
  FastDiv q1div, qdiv;
};

// dtype: 0 int32, 1 float32; op: 0 sum, 1 max.  Returns a hipError_t value.
int launch_step(const StepArgs& a, int dtype, int op, bool vec, bool nt, int grid, void* stream);
// One step as merged runs (a.run_len, a.tiles, ...): each range's blocks of a
// rank streamed as one flat space per instance.
int launch_step_merged(const StepArgs& a, int dtype, int op, bool nt, int grid, void* stream);
// Fused latency-optimal kernel; mode 1: one element per lane (contiguous
// instances), 2: any instance stride.
int launch_fused_lo(const FusedArgs& a, int P, int dtype, int op, int mode, bool nt, int grid, void* stream);
// Column-fused kernels, one instantiation per P (units written by build.py):
// bandwidth-optimal (r = 0) and shifted / latency-optimal (r >= 1), and
// their dispatcher over P = 2..128.
template <int P>
int launch_fused_bo(const ColArgs& a, int dtype, int op, bool nt, int grid, void* stream);
template <int P>
int launch_fused_mid(const ColArgs& a, int dtype, int op, bool nt, int grid, void* stream);
int launch_fused_col_any(const ColArgs& a, int P, int dtype, int op, bool nt, int grid, void* stream);
// Rank-slot kernel on flat columns (batches of short blocks, sums): the
// cyclic butterfly plans with r < L, or the Ring (ring = true); and its
// dispatcher over P = 2..128.
template <int P>
int launch_fused_rot(const ColArgs& a, int dtype, int op, bool ring, int grid, void* stream);
int launch_fused_rot_any(const ColArgs& a, int P, int dtype, int op, bool ring, int grid, void* stream);
// Column-fused kernels of the other schedules (fused_group.hip): the XOR
// group's Recursive Halving / hybrid / Recursive Doubling for P = 2..128 a
// power of two and any r, and the Ring for any P in 2..128.
int launch_fused_xor(const ColArgs& a, int P, int dtype, int op, bool nt, int grid, void* stream);
int launch_fused_ring(const ColArgs& a, int dtype, int op, bool nt, int grid, void* stream);
// Second half of a split fused launch (broadcast.hip): block b's result,
// stored on rank b by the reducing kernel, copied to the other P - 1 ranks.
int launch_broadcast(const ColArgs& a, int dtype, bool nt, int grid, void* stream);

// The same copy ordered destination by destination (broadcast.hip), for
// contiguous instances in 16-byte aligned rank buffers.  A workgroup copies
// one chunk of kStreamChunk consecutive columns of the batch's flat column
// space (the byte offset in every rank buffer is 4 * column) to one
// destination rank, one 16-byte store per thread; ids run slice by slice
// (C chunks per slice), destination by destination, chunk by chunk.
constexpr uint32_t kStreamBlock = 256;  // threads per workgroup, four columns each
constexpr uint32_t kStreamChunk = 4 * kStreamBlock;
// n / d without a branch: t = umulhi(n, mul), (t + ((n - t) >> s1)) >> s2;
// for d = 1, mul = s1 = s2 = 0 (stream_div builds it from a FastDiv).
struct StreamDiv {
  uint32_t d, mul, s1, s2;
};
inline StreamDiv stream_div(uint32_t d) {
  const FastDiv f = make_fastdiv(d);
  return f.l == 0 ? StreamDiv{d, 0, 0, 0} : StreamDiv{d, f.m, 1, f.l - 1};
}
// Host reference of the device quotient (used by the tests).
inline uint32_t stream_div_host(uint32_t n, const StreamDiv& d) {
  const uint32_t t = uint32_t((uint64_t(n) * d.mul) >> 32);
  return (t + ((n - t) >> d.s1)) >> d.s2;
}
// The scalars come first, so that a workgroup reads them in one batch of
// kernel-argument loads before it looks up its two rank pointers.
struct StreamArgs {
  uint32_t P;
  uint32_t cols;            // batch * n flat columns, < 2^32 - kStreamChunk
  uint32_t n, q, m;         // instance length, n / P, n % P
  uint32_t big;             // m * (q + 1): columns of an instance in its first m blocks (q + 1 each)
  uint32_t flat;            // 1: every column's result is on rank 0; 0: block b's on rank b (q >= kStreamChunk)
  uint32_t chunks;          // ceil(cols / kStreamChunk)
  uint32_t id0;             // id of this launch's first workgroup (a multiple of C * P)
  uint32_t regions;         // 1: XCD x takes the x-th C / X chunks of a slice; 0: every X-th chunk
  uint32_t xcd_shift;       // log2 of the XCD count X (a power of two; C is a multiple of X)
  uint32_t per_xcd;         // C / X
  StreamDiv ndiv, q1div, qdiv;  // n, q + 1, q
  StreamDiv cdiv, sdiv;     // C (a multiple of the XCD count), C * P
  void* user[kMaxP];
};
// straddle: some block or instance boundary falls inside a chunk (block
// tiles with n % P != 0 or n / P not a multiple of kStreamChunk).
int launch_broadcast_stream(const StreamArgs& a, bool nt, bool straddle, uint32_t grid, void* stream);
// Device address of the allocation-free scratch (noalloc.hip) on `device`,
// which must be the current device; looked up on the first call per device.
// Returns a hipError_t value.
int noalloc_scratch(int device, void** ptr);
// Workgroups of a step launch over `total_tiles` wave tiles, and the tile size.
int step_grid(int64_t total_tiles);
int64_t step_tile_elems();

}  // namespace ar
