// host_sanitize.cpp -- the library's host code (plan generator and C ABI)
// run on the CPU under AddressSanitizer and UndefinedBehaviorSanitizer.
//
// Built with g++ from plan.cpp and capi.cpp only: the HIP kernels are
// replaced by launchers that check the arguments the host hands them against
// what the kernels assume (rank table, template P, tile counts), and the few
// HIP runtime calls the C ABI makes are answered by a fake one-device
// runtime whose allocation, device query and launch can be made to fail.
// No device memory exists; rank "buffers" are fake addresses that the host
// code must never dereference -- AddressSanitizer stops the run if it does.
//
// Checked here, for every P in 1..128, every k in [L, 2L], the XOR group at
// power-of-two P and the Ring, over ragged, tiny and empty n:
//   - plan creation, stats and launch tables, and the launch tables replayed
//     on host rows (one heap allocation per rank and buffer, so a range that
//     strays outside its block or rank is caught) against the plain
//     definition of Allreduce (int32 sum modulo 2^32, int32 max);
//   - executes on every path, batched and strided, with the launch count
//     the stats promise and well-formed launch arguments;
//   - every documented error: bad arguments, overlapping or misaligned
//     buffers, sizes that would overflow, no device, a failed scratch
//     allocation (also on regrowth), a failed launch -- and that the plan
//     keeps working afterwards;
//   - the text dump and the timed execute, into exactly sized buffers;
//   - with "threads", the same from several threads at once (the mode for
//     ThreadSanitizer: the error text is per thread, the LDS sizes cached
//     in atomics);
//   - device scratch and timing events are freed: every fake allocation is
//     released by the time its plan is destroyed, every event by the end of
//     its execute.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <thread>
#include <vector>

#include "ar.h"
#include "ar_internal.hpp"

// ---------------------------------------------------------------------------
// Fake HIP runtime: one device, allocations that return distinct fake
// addresses (never dereferenced), failures on request.
// ---------------------------------------------------------------------------

// The state is per thread (like HIP's last error), so that several threads
// can drive the library at once; addresses come from one atomic counter.
namespace fake {
thread_local bool device_ok = true;
thread_local bool malloc_fails = false;
thread_local bool capturing = false;  // every stream reports an active graph capture
thread_local int launch_error = 0;  // hipError_t value every launcher returns when set
thread_local int last_regions = -1;  // XCD-region order of the last destination-major broadcast
thread_local int64_t live_allocs = 0, total_allocs = 0;
std::atomic<uintptr_t> next_addr{uintptr_t(1) << 44};
thread_local hipError_t last = hipSuccess;

struct Rec {
  const char* kind;
  int P, grid;
  uint32_t total_tiles;
};
thread_local std::vector<Rec> launches;
std::atomic<int> problems{0};
void problem(const char* what, int P) {
  if (problems.fetch_add(1) < 20) std::printf("LAUNCH CONTRACT: %s (P=%d)\n", what, P);
}
}  // namespace fake

hipError_t hipGetDevice(int* d) {
  if (!fake::device_ok) return fake::last = hipErrorNoDevice;
  *d = 0;
  return hipSuccess;
}
hipError_t hipSetDevice(int d) { return d == 0 ? hipSuccess : (fake::last = hipErrorInvalidDevice); }
hipError_t hipMalloc(void** p, size_t bytes) {
  if (fake::malloc_fails || bytes == 0) return fake::last = hipErrorOutOfMemory;
  *p = reinterpret_cast<void*>(fake::next_addr.fetch_add((bytes + 0xFFFF) & ~size_t(0xFFFF)));
  ++fake::live_allocs;
  ++fake::total_allocs;
  return hipSuccess;
}
hipError_t hipStreamIsCapturing(hipStream_t, hipStreamCaptureStatus* st) {
  *st = fake::capturing ? hipStreamCaptureStatusActive : hipStreamCaptureStatusNone;
  return hipSuccess;
}
// the allocation-free entry point's device array (noalloc.hip): one fake
// address, never an allocation
namespace ar {
int noalloc_scratch(int device, void** ptr) {
  *ptr = device == 0 ? reinterpret_cast<void*>(uintptr_t(1) << 42) : nullptr;
  return device == 0 ? 0 : int(hipErrorInvalidDevice);
}
}  // namespace ar
hipError_t hipFree(void* p) {
  if (p) --fake::live_allocs;
  return hipSuccess;
}
hipError_t hipGetLastError(void) {
  const hipError_t e = fake::last;
  fake::last = hipSuccess;
  return e;
}
const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "fake HIP error"; }
// Events: heap objects, so that one never destroyed is a leak; a record
// stamps the next tick of a fake clock (0.01 ms per tick).
namespace fake {
struct Event {
  int64_t stamp = -1;
};
thread_local int64_t clock = 0, live_events = 0;
thread_local bool event_fails = false;
}  // namespace fake
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned flags) {
  if (fake::event_fails) return fake::last = hipErrorOutOfMemory;
  if (flags != hipEventDisableSystemFence) return fake::last = hipErrorInvalidValue;
  *e = reinterpret_cast<hipEvent_t>(new fake::Event);
  ++fake::live_events;
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t) {
  if (!e) return fake::last = hipErrorInvalidHandle;
  reinterpret_cast<fake::Event*>(e)->stamp = ++fake::clock;
  return hipSuccess;
}
hipError_t hipEventSynchronize(hipEvent_t e) { return e ? hipSuccess : hipErrorInvalidHandle; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
  const auto* ea = reinterpret_cast<fake::Event*>(a);
  const auto* eb = reinterpret_cast<fake::Event*>(b);
  if (!ea || !eb || ea->stamp < 0 || eb->stamp < 0) return hipErrorInvalidHandle;
  *ms = float(eb->stamp - ea->stamp) * 0.01f;
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e) {
  if (!e) return hipErrorInvalidHandle;
  delete reinterpret_cast<fake::Event*>(e);
  --fake::live_events;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t attr, int device) {
  if (device != 0) return hipErrorInvalidDevice;
  if (attr == hipDeviceAttributeMaxSharedMemoryPerMultiprocessor) *v = 160 * 1024;
  else if (attr == hipDeviceAttributeMaxSharedMemoryPerBlock) *v = 64 * 1024;
  else if (attr == hipDeviceAttributeMultiprocessorCount) *v = 256;
  else return hipErrorInvalidValue;
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// Launchers: check the host's side of the kernels' contract, record, succeed.
// ---------------------------------------------------------------------------

namespace ar {

static int record(const char* kind, int P, int grid, uint32_t total_tiles) {
  if (grid < 1) fake::problem("grid below one workgroup", P);
  fake::launches.push_back({kind, P, grid, total_tiles});
  return fake::launch_error;
}

static void check_col(const ColArgs& a, int P, const char* kind) {
  if (a.P != P) fake::problem("ColArgs.P differs from the kernel's P", P);
  for (int x = 0; x < 2 * P; ++x)
    if (a.user[x] == nullptr || a.user[x] != a.user[x % P]) fake::problem("rank table not doubled", P);
  if (a.pdiv.d != uint32_t(P)) fake::problem("pdiv is not P", P);
  if (a.total_tiles == 0) fake::problem("no tiles", P);
  if (a.flat) {
    if (a.flat_cols == 0 || a.flat_cols >= 0xFFFFFFFFu - 63) fake::problem("flat column count out of range", P);
    if (a.total_tiles != (a.flat_cols + 63) / 64) fake::problem("flat tiles != ceil(cols / 64)", P);
    if (a.ndiv.d == 0 || a.q1div.d != uint32_t(a.q + 1)) fake::problem("flat divisors", P);
  } else if (a.packed) {
    if (a.ipw == 0 || a.lendiv.d == 0 || a.ipw * a.lendiv.d > 64) fake::problem("packed tile wider than a wave", P);
  } else if (a.tiles.d == 0) {
    fake::problem("no column tiles per block", P);
  }
  (void)kind;
}

template <int P>
int launch_fused_bo(const ColArgs& a, int, int, bool, int grid, void*) {
  check_col(a, P, "bo");
  if (a.r != 0) fake::problem("bandwidth-optimal kernel with r > 0", P);
  return record("fused_bo", P, grid, a.total_tiles);
}
template <int P>
int launch_fused_mid(const ColArgs& a, int, int, bool, int grid, void*) {
  check_col(a, P, "mid");
  if (a.r == 0) fake::problem("shifted kernel with r = 0", P);
  return record("fused_mid", P, grid, a.total_tiles);
}
template <int P>
int launch_fused_rot(const ColArgs& a, int, int op, bool, int grid, void*) {
  check_col(a, P, "rot");
  if (!a.flat || (op != 0 && a.r != 0 && (P < kRotMaxShiftedMinP || P > kRotMaxShiftedMaxP)))
    fake::problem("rank-slot kernel off flat columns, or a shifted max outside its P range", P);
  return record("fused_rot", P, grid, a.total_tiles);
}

// the C ABI's dispatch switches name every P in 2..128
template <int P>
void keep_launchers(std::vector<const void*>* v) {
  v->push_back(reinterpret_cast<const void*>(&launch_fused_bo<P>));
  v->push_back(reinterpret_cast<const void*>(&launch_fused_mid<P>));
  v->push_back(reinterpret_cast<const void*>(&launch_fused_rot<P>));
  if constexpr (P > 2) keep_launchers<P - 1>(v);
}

int launch_fused_xor(const ColArgs& a, int P, int, int, bool, int grid, void*) {
  check_col(a, P, "xor");
  if (P & (P - 1)) fake::problem("XOR kernel at P not a power of two", P);
  return record("fused_xor", P, grid, a.total_tiles);
}
int launch_fused_ring(const ColArgs& a, int, int, bool, int grid, void*) {
  check_col(a, a.P, "ring");
  return record("fused_ring", a.P, grid, a.total_tiles);
}
int launch_broadcast(const ColArgs& a, int, bool, int grid, void*) {
  check_col(a, a.P, "bcast");
  if (!a.split) fake::problem("broadcast without a split reduce", a.P);
  return record("broadcast", a.P, grid, a.total_tiles);
}
// The destination-major broadcast: every rank pointer 16-byte aligned, the
// column space and the chunk count consistent, a chunk spanning at most two
// roots (flat columns, or blocks of at least kStreamChunk elements), slices
// of a multiple of 8 chunks (the fake device's 256 CUs: 8 XCDs), 2048 or
// all the chunks, and a grid of whole slices below 2^32 work-items.
int launch_broadcast_stream(const StreamArgs& a, bool, bool straddle, uint32_t grid, void*) {
  const int P = int(a.P);
  if (P < 2 || P > kMaxP) fake::problem("stream broadcast P", P);
  for (int x = 0; x < P && x < kMaxP; ++x)
    if (a.user[x] == nullptr || reinterpret_cast<uintptr_t>(a.user[x]) % 16 != 0)
      fake::problem("stream broadcast rank pointer null or not 16-byte aligned", P);
  if (a.cols == 0 || uint64_t(a.cols) + kStreamChunk > UINT32_MAX) fake::problem("stream column count", P);
  if (a.chunks != (a.cols + kStreamChunk - 1) / kStreamChunk) fake::problem("stream chunk count", P);
  if (!a.flat && a.q < kStreamChunk) fake::problem("stream blocks shorter than a chunk", P);
  if (a.n == 0 || a.cols % a.n != 0 || a.ndiv.d != a.n) fake::problem("stream instance length", P);
  if (a.q != a.n / a.P || a.m != a.n % a.P || a.q1div.d != a.q + 1) fake::problem("stream block sizes", P);
  const uint32_t cmax = a.regions ? 512 : 2048;  // 256 KB / 1 MB per XCD and slice, 8 XCDs
  const uint32_t slices = (a.chunks + a.cdiv.d - 1) / std::max<uint32_t>(a.cdiv.d, 1);
  if (a.cdiv.d % 8 != 0 || a.cdiv.d > cmax || slices != (a.chunks + cmax - 1) / cmax ||
      uint64_t(a.cdiv.d) * slices >= uint64_t(a.chunks) + 8 * slices || a.sdiv.d != a.cdiv.d * a.P)
    fake::problem("stream slice size", P);
  if (a.id0 != 0 || grid != (a.chunks + a.cdiv.d - 1) / a.cdiv.d * a.sdiv.d) fake::problem("stream grid", P);
  if (a.regions > 1 || a.xcd_shift != 3 || a.per_xcd * 8 != a.cdiv.d) fake::problem("stream XCD regions", P);
  fake::last_regions = int(a.regions);
  {
    // a chunk can straddle two blocks exactly when some block or instance boundary is off the chunk grid
    bool off_grid = false;
    if (!a.flat)
      for (uint32_t b = 1; b <= a.P && !off_grid; ++b) off_grid = (b * a.q + std::min(b, a.m)) % kStreamChunk != 0;
    if (straddle != off_grid) fake::problem("stream straddle flag", P);
  }
  if (uint64_t(grid) * 256 > UINT32_MAX) fake::problem("stream grid beyond 2^32 work-items", P);
  return record("broadcast_stream", P, int(grid), a.chunks);
}
int launch_fused_lo(const FusedArgs& a, int P, int, int, int mode, bool, int grid, void*) {
  if (P < 2 || P > kFusedMaxP) fake::problem("register-resident kernel beyond its P", P);
  for (int x = 0; x < P; ++x)
    if (!a.user[x]) fake::problem("null rank pointer", P);
  if (mode < 0 || mode > 2 || a.groups < 1) fake::problem("latency-optimal mode or column groups", P);
  return record("fused_lo", P, grid, uint32_t(a.groups));
}

static void check_step(const StepArgs& a) {
  if (a.n_ranges < 1 || a.n_ranges > kMaxRanges) fake::problem("range count", a.P);
  int32_t first = 0;
  for (int i = 0; i < a.n_ranges && i < kMaxRanges; ++i) {
    const DevRange& r = a.ranges[i];
    if (r.first != first || r.count < 1 || r.count > a.P || r.p0 < 0 || r.p0 >= a.P)
      fake::problem("range table", a.P);
    for (int32_t b : {r.dst, r.own, r.dst2, r.own2, r.src})
      if ((b == kBufX || b == kBufY) && a.scratch[b - 1] == nullptr) fake::problem("scratch buffer missing", a.P);
    first += r.count;
  }
  for (int x = 0; x < a.P; ++x)
    if (!a.user[x]) fake::problem("null rank pointer", a.P);
}
int launch_step(const StepArgs& a, int, int, bool, bool, int grid, void*) {
  check_step(a);
  if (uint64_t(a.total_tiles) != uint64_t(a.P) * a.ops.d * a.batch.d * a.tps.d)
    fake::problem("step tiles != P * ops * batch * tiles per segment", a.P);
  return record("step", a.P, grid, a.total_tiles);
}
int launch_step_merged(const StepArgs& a, int, int, bool, int grid, void*) {
  check_step(a);
  uint64_t total = 0;
  for (int i = 0; i < a.n_ranges && i < kMaxRanges; ++i) {
    if (a.tile_first[i] != total) fake::problem("merged tile offsets", a.P);
    if (uint64_t(a.run_cols[i]) != uint64_t(a.batch.d) * a.run_len[i].d) fake::problem("merged columns", a.P);
    if (a.tiles[i].d != (a.run_cols[i] + 255) / 256) fake::problem("merged tiles", a.P);
    total += uint64_t(a.P) * a.tiles[i].d;
  }
  if (total != a.total_tiles) fake::problem("merged tile total", a.P);
  return record("step_merged", a.P, grid, a.total_tiles);
}
int step_grid(int64_t total_tiles) {
  const int64_t g = (total_tiles + 3) / 4;
  return int(std::min<int64_t>(std::max<int64_t>(g, 1), int64_t(1) << 22));
}
int64_t step_tile_elems() { return 256; }

}  // namespace ar

// ---------------------------------------------------------------------------
// The checks
// ---------------------------------------------------------------------------

static std::atomic<int> fails{0};
#define EXPECT(cond, ...)                                     \
  do {                                                        \
    if (!(cond)) {                                            \
      if (fails < 40) {                                       \
        std::printf("FAIL (line %d): ", __LINE__);            \
        std::printf(__VA_ARGS__);                             \
        std::printf("  [%s]\n", ar_last_error());             \
      }                                                       \
      ++fails;                                                \
    }                                                         \
  } while (0)

static int ceil_log2(int P) {
  int L = 0;
  while ((1 << L) < P) ++L;
  return L;
}

// Block b of n elements over P: the first n mod P blocks hold one more.
static void block_of(int64_t n, int P, int b, int64_t* off, int64_t* len) {
  const int64_t q = n / P, m = n % P;
  *off = b * q + std::min<int64_t>(b, m);
  *len = q + (b < m ? 1 : 0);
}

static uint32_t lcg(uint64_t* s) {
  *s = *s * 6364136223846793005ull + 1442695040888963407ull;
  return uint32_t(*s >> 33);
}

// Replays the plan's launch tables on host rows and compares every rank's
// result with the plain definition.  Rows are separate heap allocations of
// exactly n elements: an index outside a block's rank row is an ASan error.
static void replay(ar_plan* pl, int P, int64_t n, bool xorg, int op, uint64_t seed, const char* what) {
  std::vector<std::vector<int32_t*>> rows(3, std::vector<int32_t*>(P, nullptr));
  for (int buf = 0; buf < 3; ++buf)
    for (int x = 0; x < P; ++x) {
      rows[buf][x] = new int32_t[size_t(n)];
      for (int64_t e = 0; e < n; ++e) rows[buf][x][e] = buf == 0 ? int32_t(lcg(&seed)) : 0;
    }
  std::vector<int32_t> want(static_cast<size_t>(n));
  for (int64_t e = 0; e < n; ++e) {
    uint32_t s = 0;
    int32_t m = rows[0][0][e];
    for (int x = 0; x < P; ++x) {
      s += uint32_t(rows[0][x][e]);
      m = std::max(m, rows[0][x][e]);
    }
    want[size_t(e)] = op == AR_SUM ? int32_t(s) : m;
  }
  auto comb = [op](int32_t a, int32_t b) { return op == AR_SUM ? int32_t(uint32_t(a) + uint32_t(b)) : std::max(a, b); };
  int32_t nl = 0;
  ar_plan_num_launches(pl, &nl);
  for (int32_t i = 0; i < nl; ++i) {
    ar_launch_desc d;
    ar_range_desc rg[8];
    if (ar_plan_launch(pl, i, &d, rg, 8) != AR_OK || d.n_ranges > 8) {
      EXPECT(false, "%s: launch %d unreadable", what, i);
      break;
    }
    for (int j = 0; j < d.n_ranges; ++j) {
      const ar_range_desc& r = rg[j];
      EXPECT(r.src >= 0 && r.src <= 2 && r.dst >= 0 && r.dst <= 2, "%s: buffer ids", what);
      for (int c = 0; c < r.count; ++c) {
        const int p = (r.p0 + c) % P;
        for (int x = 0; x < P; ++x) {
          const int b = xorg ? (x ^ p) : ((x - p) % P + P) % P;
          const int y = xorg ? (x ^ r.delta) : ((x + r.delta) % P + P) % P;
          int64_t off, len;
          block_of(n, P, b, &off, &len);
          const int32_t* src = rows[r.src][y] + off;
          int32_t* dst = rows[r.dst][x] + off;
          if (r.kind == AR_KIND_COPY) {
            std::memmove(dst, src, size_t(len) * 4);
            continue;
          }
          std::vector<int32_t> s(src, src + len);
          const int32_t* own = rows[r.own][x] + off;
          if (r.kind == AR_KIND_REDUCE2) {
            const int32_t* own2 = rows[r.own2][x] + off;
            int32_t* dst2 = rows[r.dst2][x] + off;
            for (int64_t e = 0; e < len; ++e) dst2[e] = comb(own2[e], s[size_t(e)]);
          }
          for (int64_t e = 0; e < len; ++e) dst[e] = comb(own[e], s[size_t(e)]);
        }
      }
    }
  }
  int bad = 0;
  for (int x = 0; x < P; ++x)
    for (int64_t e = 0; e < n; ++e) bad += rows[0][x][e] != want[size_t(e)];
  EXPECT(bad == 0, "%s: %d replayed elements differ from the definition", what, bad);
  for (auto& b : rows)
    for (int32_t* r : b) delete[] r;
}

// P fake, 16-byte aligned, non-overlapping rank buffers of `bytes` each.
static std::vector<void*> fake_buffers(int P, int64_t bytes, uintptr_t base = uintptr_t(1) << 40) {
  std::vector<void*> v(static_cast<size_t>(P));
  const uintptr_t step = (uintptr_t(bytes) + 0xFFF) & ~uintptr_t(0xFFF);
  for (int x = 0; x < P; ++x) v[size_t(x)] = reinterpret_cast<void*>(base + uintptr_t(P - 1 - x) * step);
  return v;
}

static hipStream_t stream_tag() { return reinterpret_cast<hipStream_t>(uintptr_t(0x5000)); }

static void exercise(int P, int64_t n, int k, int group, int sched, int dtype, int op) {
  char what[128];
  std::snprintf(what, sizeof what, "P=%d n=%lld k=%d group=%d sched=%d dtype=%d op=%d", P, (long long)n, k, group,
                sched, dtype, op);
  ar_plan* pl = nullptr;
  ar_status st = ar_plan_create_ex(P, n, ar_dtype(dtype), ar_op(op), k, ar_group(group), ar_schedule(sched), &pl);
  EXPECT(st == AR_OK && pl, "%s: create -> %d", what, int(st));
  if (!pl) return;
  ar_stats s;
  EXPECT(ar_plan_stats(pl, &s) == AR_OK, "%s: stats", what);
  EXPECT(s.P == P && s.k == k && s.n == n && s.rs_steps + s.ag_steps == k, "%s: stats sizes", what);
  EXPECT(s.group == group && s.schedule == sched, "%s: stats group", what);
  int32_t nl = -1;
  EXPECT(ar_plan_num_launches(pl, &nl) == AR_OK && nl == s.launches, "%s: launch count", what);
  // a launch read with cap 0 writes no range
  if (nl > 0) {
    ar_launch_desc d;
    ar_range_desc guard[1];
    std::memset(guard, 0x7F, sizeof guard);
    EXPECT(ar_plan_launch(pl, 0, &d, guard, 0) == AR_OK && guard[0].p0 == 0x7F7F7F7F, "%s: cap 0 wrote", what);
    EXPECT(ar_plan_launch(pl, nl, &d, guard, 1) == AR_ERR_INVALID_ARG, "%s: launch index past the end", what);
    EXPECT(ar_plan_launch(pl, -1, &d, guard, 1) == AR_ERR_INVALID_ARG, "%s: negative launch index", what);
  }
  double t = -1;
  EXPECT(ar_plan_model_time(pl, 2e-6, 1e-10, 1e-11, &t) == AR_OK && t >= 0, "%s: model time", what);
  {  // the text dump: header, two summary lines and one line per launch, into exactly sized buffers
    int64_t len = -1, len2 = -1;
    EXPECT(ar_plan_dump(pl, nullptr, 0, &len) == AR_OK && len > 0, "%s: dump length", what);
    char* full = new char[size_t(len) + 1];
    EXPECT(ar_plan_dump(pl, full, len + 1, &len2) == AR_OK && len2 == len && int64_t(std::strlen(full)) == len,
           "%s: dump", what);
    EXPECT(std::count(full, full + len, '\n') == 3 + nl, "%s: dump lines", what);
    char* part = new char[7];
    EXPECT(ar_plan_dump(pl, part, 7, &len2) == AR_OK && std::strlen(part) == 6 && std::strncmp(part, full, 6) == 0,
           "%s: truncated dump", what);
    delete[] full;
    delete[] part;
  }
  if (n > 0 && n <= 4 * P + 8 && dtype == AR_INT32) replay(pl, P, n, group == AR_GROUP_XOR, op, uint64_t(P) * 7919 + k, what);

  // executes on every path; the fake buffers are never dereferenced
  for (int path : {AR_PATH_AUTO, AR_PATH_STEPWISE, AR_PATH_FUSED}) {
    const ar_status ps = ar_plan_set_path(pl, ar_path(path));
    if (P == 1 && path == AR_PATH_FUSED) {
      EXPECT(ps == AR_ERR_UNSUPPORTED, "%s: fused path at P = 1", what);
      continue;
    }
    EXPECT(ps == AR_OK, "%s: set path %d", what, path);
    for (int64_t batch : {int64_t(1), int64_t(3)}) {
      const int64_t stride = n + 5;
      std::vector<void*> bufs = fake_buffers(P, ((batch - 1) * stride + n) * 4 + 64);
      fake::launches.clear();
      st = ar_execute_batched(pl, bufs.data(), batch, stride, stream_tag());
      EXPECT(st == AR_OK, "%s: execute path %d batch %lld -> %d", what, path, (long long)batch, int(st));
      const bool fused = path == AR_PATH_FUSED || (path == AR_PATH_AUTO && s.fused_ok);
      const size_t expect = (n == 0 || P == 1) ? 0 : fused ? size_t(s.fused_launches) : size_t(nl);
      EXPECT(fake::launches.size() == expect, "%s: path %d made %zu launches, stats say %zu", what, path,
             fake::launches.size(), expect);
      // the timed execute: one duration per launch, into an exactly sized array (cap may be short)
      const int32_t cap = int32_t(std::min<size_t>(expect, 3));
      float* ms = new float[size_t(cap) + (cap == 0)];
      int32_t got = -1;
      fake::launches.clear();
      st = ar_execute_timed(pl, bufs.data(), batch, stride, stream_tag(), cap ? ms : nullptr, cap, &got);
      EXPECT(st == AR_OK && got == int32_t(expect) && fake::launches.size() == expect, "%s: timed execute", what);
      for (int32_t i = 0; i < cap; ++i) EXPECT(ms[i] > 0.0f, "%s: launch %d timed at %g ms", what, i, ms[i]);
      EXPECT(fake::live_events == 0, "%s: %lld events left", what, (long long)fake::live_events);
      delete[] ms;
    }
  }
  ar_plan_destroy(pl);
  EXPECT(fake::live_allocs == 0, "%s: scratch not freed (%lld live)", what, (long long)fake::live_allocs);
}

// Which broadcast a split plan takes: the destination-major one for
// contiguous instances in 16-byte aligned buffers, on flat columns at any P
// or on blocks of at least kStreamChunk elements in rank spans of at least
// 2 MiB; the tiled one otherwise.  On flat columns its chunks go in XCD
// regions above 16 MiB per rank, interleaved up to it.
struct BcastCase {
  int P;
  int64_t n;
  int k, group, batch;
  int64_t stride_extra;
  uintptr_t misalign;
  const char* expect;
  int regions;  // the destination-major copy's chunk order: 1 XCD regions, 0 interleaved, -1 tiled copy
};

static void check_broadcast_case(const BcastCase& c);

static void broadcast_choice() {
  const BcastCase cases[] = {
      {127, int64_t(1) << 26, 14, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 0},
      {127, int64_t(1) << 25, 14, AR_GROUP_CYCLIC, 2, 0, 0, "broadcast_stream", 1},   // rank slots below 256 MiB per instance: flat, regions
      {37, int64_t(1) << 22, 12, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 0},    // flat, exactly 16 MiB: interleaved
      {37, (int64_t(1) << 22) + 1024, 12, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 1},  // just above: regions
      {127, int64_t(1) << 26, 14, AR_GROUP_CYCLIC, 3, 5, 0, "broadcast", -1},          // gaps between instances
      {127, int64_t(1) << 26, 14, AR_GROUP_CYCLIC, 1, 0, 4, "broadcast", -1},          // a rank buffer off 16 bytes
      {127, int64_t(1) << 25, 14, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 1},   // 128 MiB per rank: XCD regions
      {127, int64_t(1) << 24, 14, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 1},   // 64 MiB
      {127, (int64_t(1) << 24) - 1024, 14, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 1},
      {127, int64_t(1) << 19, 14, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 0},   // 2 MiB per rank: flat, interleaved
      {127, (int64_t(1) << 19) - 1024, 14, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 0},
      {64, int64_t(1) << 19, 12, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 0},
      {100, int64_t(1) << 25, 14, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 1},
      {104, int64_t(1) << 24, 14, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 1},
      {64, int64_t(1) << 24, 12, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 1},     // blocks on the chunk grid: regions
      {127, 1024 * 127 + 333, 14, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 0},
      {64, int64_t(1) << 26, 12, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 1},
      {128, int64_t(1) << 26, 14, AR_GROUP_XOR, 1, 0, 0, "broadcast_stream", 1},
      {128, int64_t(1) << 21, 14, AR_GROUP_XOR, 1, 0, 0, "broadcast_stream", 0},      // XOR sums on flat columns: 8 MiB
      {64, int64_t(1) << 22, 12, AR_GROUP_XOR, 1, 0, 0, "broadcast_stream", 0},       // 16 MiB: interleaved
      {64, int64_t(1) << 23, 12, AR_GROUP_XOR, 1, 0, 0, "broadcast_stream", 1},       // 32 MiB: regions
      {32, int64_t(1) << 24, 10, AR_GROUP_XOR, 1, 0, 0, "broadcast_stream", 1},       // gradient-sync shape, 64 MiB
      {127, 2304, 14, AR_GROUP_CYCLIC, 8, 0, 0, "broadcast_stream", 0},                // flat columns, root rank 0
      {127, 2304, 14, AR_GROUP_CYCLIC, 8, 3, 0, "broadcast", -1},
      {128, 2304, 14, AR_GROUP_XOR, 4, 0, 0, "broadcast_stream", 0},
      {48, 2304, 12, AR_GROUP_CYCLIC, 8, 0, 0, "broadcast_stream", 0},                  // flat, any P
      {48, 2304, 12, AR_GROUP_CYCLIC, 8192, 0, 0, "broadcast_stream", 1},               // flat, 72 MiB per rank: regions
      {127, 2304, 14, AR_GROUP_CYCLIC, 60000, 0, 0, "broadcast", -1},                   // grid above 2^32 work-items
      {127, 2304, 14, AR_GROUP_CYCLIC, 56000, 0, 0, "broadcast_stream", 1},            // just below it
  };
  for (const BcastCase& c : cases) check_broadcast_case(c);
}

static void check_broadcast_case(const BcastCase& c) {
  ar_plan* pl = nullptr;
  EXPECT(ar_plan_create_ex(c.P, c.n, AR_FLOAT32, AR_SUM, c.k, ar_group(c.group), AR_SCHEDULE_BUTTERFLY, &pl) ==
             AR_OK, "broadcast choice: create P=%d n=%lld", c.P, (long long)c.n);
  if (!pl) return;
  ar_stats s;
  EXPECT(ar_plan_stats(pl, &s) == AR_OK && s.fused_launches == 2, "broadcast choice: P=%d n=%lld not split", c.P,
         (long long)c.n);
  const int64_t stride = c.n + c.stride_extra;
  std::vector<void*> bufs = fake_buffers(c.P, ((c.batch - 1) * stride + c.n) * 4 + 64);
  bufs[size_t(c.P / 2)] = reinterpret_cast<char*>(bufs[size_t(c.P / 2)]) + c.misalign;
  fake::launches.clear();
  fake::last_regions = -1;
  EXPECT(ar_execute_batched(pl, bufs.data(), c.batch, stride, stream_tag()) == AR_OK && fake::launches.size() == 2 &&
             std::strcmp(fake::launches[1].kind, c.expect) == 0 && fake::last_regions == c.regions,
         "broadcast choice: P=%d n=%lld batch %d stride +%lld misalign %zu took %s, expected %s", c.P,
         (long long)c.n, c.batch, (long long)c.stride_extra, size_t(c.misalign),
         fake::launches.size() == 2 ? fake::launches[1].kind : "?", c.expect);
  ar_plan_destroy(pl);
}

// Block tiles (AR_FUSED_ROTATE=0) whose blocks all start on the chunk grid:
// XCD regions from 104 ranks or from 32 MiB per rank, interleaved chunks
// below.  Plans read the variable when they are created: single-threaded
// only.
static void broadcast_block_order() {
  const BcastCase cases[] = {
      {128, int64_t(1) << 21, 14, AR_GROUP_XOR, 1, 0, 0, "broadcast_stream", 1},      // P >= 104: regions
      {64, int64_t(1) << 22, 12, AR_GROUP_XOR, 1, 0, 0, "broadcast_stream", 0},       // 16 MiB: interleaved
      {64, int64_t(1) << 23, 12, AR_GROUP_XOR, 1, 0, 0, "broadcast_stream", 1},       // 32 MiB: regions
      {32, int64_t(1) << 24, 10, AR_GROUP_XOR, 1, 0, 0, "broadcast_stream", 1},       // 64 MiB
      {64, int64_t(1) << 22, 12, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 0},    // cyclic, 16 MiB
      {64, int64_t(1) << 24, 12, AR_GROUP_CYCLIC, 1, 0, 0, "broadcast_stream", 1},    // cyclic, 64 MiB
  };
  setenv("AR_FUSED_ROTATE", "0", 1);
  for (const BcastCase& c : cases) check_broadcast_case(c);
  unsetenv("AR_FUSED_ROTATE");
}

// AR_BCAST_STREAM = 2 / 3: the destination-major copy with interleaved chunks
// / XCD regions wherever the call allows it, whatever the size; 1 with the
// order by size; 0 the tiled copy.  Plans read the variable when they are
// created: single-threaded only.
static void broadcast_order_override() {
  struct Case {
    int P;
    int64_t n;
    int batch;
    const char* env;
    const char* expect;
    int regions;
  };
  const Case cases[] = {
      {127, int64_t(1) << 26, 1, "2", "broadcast_stream", 0}, {127, int64_t(1) << 26, 1, "3", "broadcast_stream", 1},
      {127, int64_t(1) << 26, 1, "1", "broadcast_stream", 0}, {127, 127 * 1024 + 77, 1, "1", "broadcast_stream", 0},
      {127, 127 * 1024 + 77, 1, "2", "broadcast_stream", 0},  {127, 127 * 1024 + 77, 1, "3", "broadcast_stream", 1},
      {127, 127 * 1024 + 77, 1, "0", "broadcast", -1},         {127, 2304, 8, "1", "broadcast_stream", 0},
      {127, 2304, 8, "3", "broadcast_stream", 1},              {48, 2304, 8, "2", "broadcast_stream", 0},
      {127, 127 * 1024 + 77, 1, "7", "broadcast_stream", 0},   // not a mode: the default rules (flat columns)
  };
  for (const Case& c : cases) {
    setenv("AR_BCAST_STREAM", c.env, 1);
    ar_plan* pl = nullptr;
    EXPECT(ar_plan_create_ex(c.P, c.n, AR_FLOAT32, AR_SUM, c.P == 48 ? 12 : 14, AR_GROUP_CYCLIC,
                             AR_SCHEDULE_BUTTERFLY, &pl) == AR_OK,
           "broadcast order: create P=%d n=%lld", c.P, (long long)c.n);
    unsetenv("AR_BCAST_STREAM");
    if (!pl) continue;
    ar_stats st;
    EXPECT(ar_plan_stats(pl, &st) == AR_OK && st.fused_bcast_stream == (c.regions >= 0 ? 1 : 0),
           "broadcast order: stats P=%d n=%lld env %s", c.P, (long long)c.n, c.env);
    std::vector<void*> bufs = fake_buffers(c.P, c.batch * c.n * 4 + 64);
    fake::launches.clear();
    fake::last_regions = -1;
    EXPECT(ar_execute_batched(pl, bufs.data(), c.batch, c.n, stream_tag()) == AR_OK && fake::launches.size() == 2 &&
               std::strcmp(fake::launches[1].kind, c.expect) == 0 && fake::last_regions == c.regions,
           "broadcast order: P=%d n=%lld batch %d env %s took %s (regions %d), expected %s (%d)", c.P,
           (long long)c.n, c.batch, c.env, fake::launches.size() == 2 ? fake::launches[1].kind : "?",
           fake::last_regions, c.expect, c.regions);
    ar_plan_destroy(pl);
  }
}

static void errors() {
  ar_plan* pl = nullptr;
  EXPECT(ar_plan_create(4, 100, AR_FLOAT32, AR_SUM, 2, nullptr) == AR_ERR_INVALID_ARG, "null out_plan");
  EXPECT(ar_plan_create(0, 100, AR_FLOAT32, AR_SUM, 0, &pl) == AR_ERR_INVALID_ARG && !pl, "P = 0");
  EXPECT(ar_plan_create(129, 100, AR_FLOAT32, AR_SUM, 8, &pl) == AR_ERR_UNSUPPORTED, "P = 129");
  EXPECT(ar_plan_create(5, -1, AR_FLOAT32, AR_SUM, 4, &pl) == AR_ERR_INVALID_ARG, "n = -1");
  EXPECT(ar_plan_create(5, (int64_t(1) << 46) + 1, AR_FLOAT32, AR_SUM, 4, &pl) == AR_ERR_INVALID_ARG, "n > 2^46");
  EXPECT(ar_plan_create(5, INT64_MAX, AR_FLOAT32, AR_SUM, 4, &pl) == AR_ERR_INVALID_ARG, "n = INT64_MAX");
  EXPECT(ar_plan_create(5, 100, AR_FLOAT32, AR_SUM, 2, &pl) == AR_ERR_INVALID_ARG, "k below L");
  EXPECT(ar_plan_create(5, 100, AR_FLOAT32, AR_SUM, 7, &pl) == AR_ERR_INVALID_ARG, "k above 2L");
  EXPECT(ar_plan_create(5, 100, ar_dtype(7), AR_SUM, 4, &pl) == AR_ERR_UNSUPPORTED, "dtype");
  EXPECT(ar_plan_create(5, 100, AR_FLOAT32, ar_op(9), 4, &pl) == AR_ERR_UNSUPPORTED, "op");
  EXPECT(ar_plan_create_ex(6, 100, AR_FLOAT32, AR_SUM, 4, AR_GROUP_XOR, AR_SCHEDULE_BUTTERFLY, &pl) ==
             AR_ERR_INVALID_ARG, "XOR at P = 6");
  EXPECT(ar_plan_create_ex(8, 100, AR_FLOAT32, AR_SUM, 14, AR_GROUP_XOR, AR_SCHEDULE_RING, &pl) == AR_ERR_INVALID_ARG,
         "Ring over XOR");
  EXPECT(ar_plan_create_ex(5, 100, AR_FLOAT32, AR_SUM, 7, AR_GROUP_CYCLIC, AR_SCHEDULE_RING, &pl) ==
             AR_ERR_INVALID_ARG, "Ring k");
  EXPECT(ar_plan_create_ex(5, 100, AR_FLOAT32, AR_SUM, 4, ar_group(3), AR_SCHEDULE_BUTTERFLY, &pl) ==
             AR_ERR_INVALID_ARG, "group");
  EXPECT(ar_plan_create_ex(5, 100, AR_FLOAT32, AR_SUM, 4, AR_GROUP_CYCLIC, ar_schedule(3), &pl) == AR_ERR_INVALID_ARG,
         "schedule");
  EXPECT(pl == nullptr, "a failed create set the plan");
  for (int sv = -1; sv <= 9; ++sv) EXPECT(ar_status_string(ar_status(sv)) != nullptr, "status string %d", sv);

  ar_stats s;
  int32_t k = 0;
  double tau = 0, rc = 0;
  EXPECT(ar_plan_stats(nullptr, &s) == AR_ERR_INVALID_ARG, "stats of NULL");
  {
    ar_plan* p3 = nullptr;
    int64_t len = 0;
    char b[4];
    float ms[2];
    int32_t got = 0;
    void* bufs3[3] = {reinterpret_cast<void*>(0x10000), reinterpret_cast<void*>(0x20000), reinterpret_cast<void*>(0x30000)};
    EXPECT(ar_plan_create(3, 8, AR_INT32, AR_SUM, 2, &p3) == AR_OK, "create P=3");
    EXPECT(ar_plan_dump(nullptr, b, 4, &len) == AR_ERR_INVALID_ARG, "dump of NULL");
    EXPECT(ar_plan_dump(p3, b, 4, nullptr) == AR_ERR_INVALID_ARG, "dump without len");
    EXPECT(ar_plan_dump(p3, b, -1, &len) == AR_ERR_INVALID_ARG, "dump cap < 0");
    EXPECT(ar_plan_dump(p3, nullptr, 4, &len) == AR_ERR_INVALID_ARG, "dump NULL buf with cap");
    EXPECT(ar_execute_timed(p3, bufs3, 1, 8, nullptr, ms, 2, nullptr) == AR_ERR_INVALID_ARG, "timed without count");
    EXPECT(ar_execute_timed(p3, bufs3, 1, 8, nullptr, ms, -1, &got) == AR_ERR_INVALID_ARG, "timed cap < 0");
    EXPECT(ar_execute_timed(p3, bufs3, 1, 8, nullptr, nullptr, 2, &got) == AR_ERR_INVALID_ARG, "timed NULL array");
    EXPECT(ar_execute_timed(nullptr, bufs3, 1, 8, nullptr, ms, 2, &got) == AR_ERR_INVALID_ARG, "timed NULL plan");
    ar_plan_destroy(p3);
  }
  EXPECT(ar_plan_set_path(nullptr, AR_PATH_AUTO) == AR_ERR_INVALID_ARG, "path of NULL");
  EXPECT(ar_execute(nullptr, nullptr, nullptr) == AR_ERR_INVALID_ARG, "execute NULL");
  EXPECT(ar_model_time(0, 1e6, 0, 1, 1, 1, &tau) == AR_ERR_INVALID_ARG, "model P = 0");
  EXPECT(ar_model_time(8, -1, 4, 1, 1, 1, &tau) == AR_ERR_INVALID_ARG, "model m < 0");
  EXPECT(ar_model_time(8, 1e6, 4, 1, 1, 1, nullptr) == AR_ERR_INVALID_ARG, "model NULL");
  EXPECT(ar_model_best_k(8, 1e6, 1, 1, 1, nullptr, &rc) == AR_ERR_INVALID_ARG, "best k NULL");
  for (int P = 1; P <= 128; ++P)
    for (double m : {0.0, 1.0, 4e3, 1e9}) {
      EXPECT(ar_model_best_k(P, m, 3e-6, 1e-10, 1e-11, &k, &rc) == AR_OK && k >= ceil_log2(P) && k <= 2 * ceil_log2(P),
             "best k P=%d", P);
      EXPECT(ar_model_best_k(P, m, 3e-6, 1e-10, 1e-11, &k, nullptr) == AR_OK, "best k without r* P=%d", P);
    }
  ar_plan_destroy(nullptr);
}

static void execute_errors() {
  // P = 7, k = 5: r = 1, the step-wise path needs scratch
  ar_plan* pl = nullptr;
  const int64_t n = 1000;
  EXPECT(ar_plan_create(7, n, AR_FLOAT32, AR_SUM, 5, &pl) == AR_OK, "create P=7 k=5");
  if (!pl) return;
  ar_plan_set_path(pl, AR_PATH_STEPWISE);
  std::vector<void*> bufs = fake_buffers(7, n * 4);
  // argument errors, before any device work
  fake::launches.clear();
  EXPECT(ar_execute(pl, nullptr, stream_tag()) == AR_ERR_INVALID_ARG, "NULL table");
  EXPECT(ar_execute_batched(pl, bufs.data(), 0, n, stream_tag()) == AR_ERR_INVALID_ARG, "batch 0");
  EXPECT(ar_execute_batched(pl, bufs.data(), 2, n - 1, stream_tag()) == AR_ERR_INVALID_ARG, "stride < n");
  std::vector<void*> bad = bufs;
  bad[3] = nullptr;
  EXPECT(ar_execute(pl, bad.data(), stream_tag()) == AR_ERR_INVALID_ARG, "NULL rank");
  bad = bufs;
  bad[3] = static_cast<char*>(bad[3]) + 2;
  EXPECT(ar_execute(pl, bad.data(), stream_tag()) == AR_ERR_INVALID_ARG, "misaligned rank");
  bad = bufs;
  bad[5] = static_cast<char*>(bad[2]) + (n - 1) * 4;
  EXPECT(ar_execute(pl, bad.data(), stream_tag()) == AR_ERR_ALIAS, "overlapping ranks");
  bad = bufs;
  bad[6] = bad[0];
  EXPECT(ar_execute(pl, bad.data(), stream_tag()) == AR_ERR_ALIAS, "same rank twice");
  // sizes whose byte extent would overflow 64-bit arithmetic
  EXPECT(ar_execute_batched(pl, bufs.data(), int64_t(1) << 40, int64_t(1) << 30, stream_tag()) == AR_ERR_INVALID_ARG,
         "batch * stride overflow");
  EXPECT(ar_execute_batched(pl, bufs.data(), INT64_MAX, n, stream_tag()) == AR_ERR_INVALID_ARG, "batch = INT64_MAX");
  EXPECT(ar_execute_batched(pl, bufs.data(), 2, INT64_MAX, stream_tag()) == AR_ERR_INVALID_ARG, "stride = INT64_MAX");
  EXPECT(fake::launches.empty() && fake::total_allocs == 0, "device work before the arguments were checked");

  // no device
  fake::device_ok = false;
  EXPECT(ar_execute(pl, bufs.data(), stream_tag()) == AR_ERR_NO_DEVICE, "no device");
  fake::device_ok = true;
  // scratch allocation fails: nothing launched, the plan still works afterwards
  fake::malloc_fails = true;
  EXPECT(ar_execute(pl, bufs.data(), stream_tag()) == AR_ERR_OUT_OF_MEMORY, "scratch allocation failure");
  EXPECT(fake::launches.empty() && fake::live_allocs == 0, "launched or kept memory after a failed allocation");
  fake::malloc_fails = false;
  EXPECT(ar_execute(pl, bufs.data(), stream_tag()) == AR_OK && fake::live_allocs == 1, "execute after the failure");
  // regrowth for a larger batch fails: the error is reported and the old
  // scratch stays (graphs captured earlier may address it)
  std::vector<void*> big = fake_buffers(7, 4 * n * 4);
  fake::malloc_fails = true;
  EXPECT(ar_execute_batched(pl, big.data(), 4, n, stream_tag()) == AR_ERR_OUT_OF_MEMORY, "regrowth failure");
  EXPECT(fake::live_allocs == 1, "old scratch released after a failed regrowth");
  fake::malloc_fails = false;
  // regrowth while the stream is being captured: refused before any launch
  // or allocation; a call that fits the scratch may be captured
  fake::capturing = true;
  fake::launches.clear();
  EXPECT(ar_execute_batched(pl, big.data(), 4, n, stream_tag()) == AR_ERR_UNSUPPORTED, "regrowth under capture");
  EXPECT(fake::launches.empty() && fake::live_allocs == 1, "work or allocation after a refused capture");
  EXPECT(ar_execute(pl, bufs.data(), stream_tag()) == AR_OK, "capture without regrowth");
  fake::capturing = false;
  EXPECT(ar_execute_batched(pl, big.data(), 4, n, stream_tag()) == AR_OK && fake::live_allocs == 2,
         "regrowth keeps the old scratch until destroy");
  // a smaller call reuses the scratch
  const int64_t before = fake::total_allocs;
  EXPECT(ar_execute(pl, bufs.data(), stream_tag()) == AR_OK && fake::total_allocs == before, "scratch reuse");
  // the allocation-free entry point: no allocation, the library's array as X / Y
  {
    const int64_t allocs = fake::total_allocs, live = fake::live_allocs;
    fake::launches.clear();
    fake::malloc_fails = true;  // any allocation attempt would fail the call
    EXPECT(ar_execute_noalloc(pl, big.data(), 4, n, stream_tag()) == AR_OK && !fake::launches.empty(),
           "allocation-free execute");
    EXPECT(ar_execute_noalloc(pl, bufs.data(), 1, n, stream_tag()) == AR_OK, "allocation-free, smaller call");
    fake::malloc_fails = false;
    EXPECT(fake::total_allocs == allocs && fake::live_allocs == live, "the allocation-free execute allocated");
    // beyond the array: 2 * 7 * round64(extent) * 4 bytes > 64 MiB
    const int64_t many = (int64_t(64) << 20) / (2 * 7 * 4 * n) + 2;
    std::vector<void*> huge = fake_buffers(7, many * n * 4);
    fake::launches.clear();
    EXPECT(ar_execute_noalloc(pl, huge.data(), many, n, stream_tag()) == AR_ERR_UNSUPPORTED &&
               fake::launches.empty(), "allocation-free execute beyond the array");
    EXPECT(std::strstr(ar_last_error_message(), "at most") != nullptr, "no size in the message");
  }
  // growth one batch at a time: the scratch at least doubles, so batches 1..16
  // allocate five buffers (1, 2, 4, 8 and 16 instances' worth), all kept until destroy
  {
    ar_plan* g = nullptr;
    EXPECT(ar_plan_create(7, n, AR_FLOAT32, AR_SUM, 5, &g) == AR_OK, "create for growth");
    ar_plan_set_path(g, AR_PATH_STEPWISE);
    std::vector<void*> b16 = fake_buffers(7, 16 * n * 4, uintptr_t(1) << 43);
    const int64_t a0 = fake::total_allocs, l0 = fake::live_allocs;
    for (int64_t batch = 1; batch <= 16; ++batch)
      EXPECT(ar_execute_batched(g, b16.data(), batch, n, stream_tag()) == AR_OK, "growth batch %lld", (long long)batch);
    EXPECT(fake::total_allocs - a0 == 5 && fake::live_allocs - l0 == 5, "growth allocated %lld buffers",
           (long long)(fake::total_allocs - a0));
    ar_plan_destroy(g);
    EXPECT(fake::live_allocs == l0, "growth buffers not freed by destroy");
  }
  // a failed launch is reported as a HIP error and stops the execute
  fake::launches.clear();
  fake::launch_error = int(hipErrorLaunchFailure);
  EXPECT(ar_execute(pl, bufs.data(), stream_tag()) == AR_ERR_HIP && fake::launches.size() == 1, "launch failure");
  EXPECT(std::strlen(ar_last_error()) > 0, "no message for the launch failure");
  ar_plan_set_path(pl, AR_PATH_FUSED);
  EXPECT(ar_execute(pl, bufs.data(), stream_tag()) == AR_ERR_HIP, "fused launch failure");
  fake::launch_error = 0;
  EXPECT(ar_execute(pl, bufs.data(), stream_tag()) == AR_OK, "execute after the launch failure");
  // a timing event that cannot be created is reported, and no event is left behind
  fake::event_fails = true;
  float ms[8];
  int32_t got = -1;
  EXPECT(ar_execute_timed(pl, bufs.data(), 1, n, stream_tag(), ms, 8, &got) == AR_ERR_HIP && got == 0,
         "event failure");
  fake::event_fails = false;
  EXPECT(fake::live_events == 0, "events left after a failure");
  EXPECT(ar_execute_timed(pl, bufs.data(), 1, n, stream_tag(), ms, 8, &got) == AR_OK && got == 1, "timed fused");
  ar_plan_destroy(pl);
  EXPECT(fake::live_allocs == 0, "scratch not freed by destroy");
  // n = 0: nothing is touched, NULL pointers allowed
  EXPECT(ar_plan_create(9, 0, AR_INT32, AR_MAX, 5, &pl) == AR_OK, "create n = 0");
  std::vector<void*> nulls(9, nullptr);
  fake::launches.clear();
  EXPECT(ar_execute(pl, nulls.data(), stream_tag()) == AR_OK && fake::launches.empty(), "n = 0 execute");
  ar_plan_destroy(pl);
}

// Every plan of P = first, first + step, ... up to pmax.
static int sweep(int first, int step, int pmax) {
  int plans = 0;
  for (int P = first; P <= pmax; P += step) {
    const int L = ceil_log2(P);
    const bool pow2 = (P & (P - 1)) == 0;
    std::vector<int64_t> ns = {0, 1, 3 * int64_t(P) + 2, 64 * int64_t(P) + 5, int64_t(1) << 22};
    if (P > 2) ns.push_back(P - 1);
    for (int k = L; k <= 2 * L; ++k)
      for (size_t i = 0; i < ns.size(); ++i) {
        const int op = (P + k + int(i)) % 2;  // int32 sum and max alternate
        exercise(P, ns[i], k, AR_GROUP_CYCLIC, AR_SCHEDULE_BUTTERFLY, AR_INT32, op);
        if (pow2) exercise(P, ns[i], k, AR_GROUP_XOR, AR_SCHEDULE_BUTTERFLY, AR_INT32, op);
        if (i == 2) exercise(P, ns[i], k, AR_GROUP_CYCLIC, AR_SCHEDULE_BUTTERFLY, AR_FLOAT32, AR_SUM);
        plans += 1 + pow2 + (i == 2);
      }
    for (size_t i = 0; i < ns.size(); ++i) {
      exercise(P, ns[i], 2 * (P - 1), AR_GROUP_CYCLIC, AR_SCHEDULE_RING, AR_INT32, AR_SUM);
      ++plans;
    }
  }
  return plans;
}

// argv: [pmax] runs everything on one thread; "threads" T pmax runs the
// error checks and the sweep on T threads at once (P dealt out round robin),
// the mode for ThreadSanitizer.
int main(int argc, char** argv) {
  std::vector<const void*> keep;
  ar::keep_launchers<128>(&keep);
  int plans = 0;
  if (argc > 1 && std::strcmp(argv[1], "threads") == 0) {
    const int nt = argc > 2 ? std::atoi(argv[2]) : 8;
    const int pmax = argc > 3 ? std::atoi(argv[3]) : 40;
    std::vector<std::thread> th;
    std::vector<int> counts(size_t(nt), 0);
    th.emplace_back([] {
      errors();
      execute_errors();
      broadcast_choice();
    });
    for (int t = 0; t < nt; ++t) th.emplace_back([t, nt, pmax, &counts] { counts[size_t(t)] = sweep(1 + t, nt, pmax); });
    for (std::thread& x : th) x.join();
    for (int c : counts) plans += c;
  } else {
    const int pmax = argc > 1 ? std::atoi(argv[1]) : 128;
    errors();
    execute_errors();
    broadcast_choice();
    broadcast_order_override();
    broadcast_block_order();
    plans = sweep(1, 1, pmax);
  }
  std::printf("%d plans, %d launch contract problems, %d failures\n", plans, fake::problems.load(), fails.load());
  return (fails || fake::problems) ? 1 : 0;
}
