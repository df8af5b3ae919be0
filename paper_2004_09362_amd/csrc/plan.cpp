// plan.cpp -- host-side schedule generator for the generalized Allreduce.
//
// Kolmakov & Zhang, "A Generalization of the Allreduce Operation"
// (arXiv:2004.09362).  Vocabulary: the distributed vector t^p q is called
// "placement p"; with the cyclic group t_k(x) = x + k and h = identity, rank
// x holds block (x - p) mod P of it (Sec. 5.1-5.2).  A step with operator
// t^{-f} moves placement p + f of rank x + f onto placement p of rank x
// (Sec. 5.3): the same block, so every pull reads the peer's buffer at the
// block offset the receiver writes (no data shift, Sec. 7).
//
// Reduction phase (Sec. 7): N_0 = P, f_i = floor(N_i/2), c_i = ceil(N_i/2),
// N_{i+1} = c_i; step i combines placements [c_i - f_i, c_i) with the
// received [c_i, N_i).  Shifted by s = 0 .. w-1 (Sec. 8; w = min(2^r, P))
// the kept placements become s + [1, c_i) for the primed partial sums q' and
// s itself for the starred q* (which skips odd steps).  Primed sums at one
// placement are the same whichever shift reaches them, so each is computed
// once; starred ones are kept apart from primed ones once an odd step has
// made them differ (Sec. 9).
//
// Buffers.  r = 0: everything runs in place in the caller's buffers U (the
// written placements [c-f, c) never meet the ones peers read, [c, N)).
// r > 0: primed sums ping-pong between two scratch buffers X and Y because
// peers read placements that are also rewritten in the same step; starred
// sums live in U once they differ from the primed ones (peers never read
// them), and share the primed storage until then.
//
// Distribution phase (Sec. 7, reversed steps without combination): with
// placements [0, h) held, the reversed step i fetches [max(c_i, h), N_i)
// from rank x - f_i, only when N_i > h; exactly L - r steps remain.
//
// Group of Table 1b (power-of-two P, t_k(x) = x XOR k; every element is its
// own inverse).  Placement p of rank x holds block x XOR p, and a step with
// operator t_f pulls from rank x XOR f.  N_i = P / 2^i, f_i = c_i = N_i / 2.
// The shifts s < w form a subgroup, so shifting the schedule by s only
// permutes its vectors: while f_i >= w the w shifted schedules are one and
// the same, and step i combines placements [0, f_i) with the received
// [f_i, 2 f_i) in place (Recursive Halving, Sec. 7); once f_i < w every one
// of the w held placements combines with its partner's (Recursive
// Doubling, Sec. 9), ping-ponging through scratch since peers read what is
// rewritten.  The last of those steps writes the caller's buffers.  The
// distribution fetches [f_i, 2 f_i) from rank x XOR f_i for the L - r steps
// with 2 f_i > w.
//
// Ring (Sec. 6, cyclic group): P - 1 reduction steps, each combining
// placement i + 1 with placement i of rank x - 1 (one block, in place), then
// P - 1 distribution steps copying placement j - 1 of rank x - 1 to
// placement j.
#include <algorithm>
#include <cstdio>
#include <set>
#include <string>
#include <vector>

#include "ar_internal.hpp"

namespace ar {

static int32_t ceil_log2(int32_t P) {
  int32_t L = 0;
  while ((int64_t(1) << L) < P) ++L;
  return L;
}

static int32_t pmod(int64_t a, int32_t P) {
  int64_t v = a % P;
  return int32_t(v < 0 ? v + P : v);
}

namespace {

struct POp {
  int32_t kind, delta, dst, own, dst2, own2, src;
  bool same(const POp& o) const {
    return kind == o.kind && delta == o.delta && dst == o.dst && own == o.own && dst2 == o.dst2 &&
           own2 == o.own2 && src == o.src;
  }
};

// Group per-placement operations into maximal runs of consecutive placements.
void emit_launch(std::vector<Launch>* out, int32_t phase, const std::vector<std::vector<POp>>& per_p) {
  Launch l;
  l.phase = phase;
  const int32_t P = int32_t(per_p.size());
  std::vector<std::vector<bool>> used(P);
  for (int32_t p = 0; p < P; ++p) used[p].assign(per_p[p].size(), false);
  for (int32_t p = 0; p < P; ++p) {
    for (size_t i = 0; i < per_p[p].size(); ++i) {
      if (used[p][i]) continue;
      const POp& op = per_p[p][i];
      used[p][i] = true;
      int32_t count = 1;
      for (int32_t q = p + 1; q < P; ++q) {
        bool found = false;
        for (size_t j = 0; j < per_p[q].size(); ++j) {
          if (!used[q][j] && per_p[q][j].same(op)) {
            used[q][j] = true;
            found = true;
            break;
          }
        }
        if (!found) break;
        ++count;
      }
      l.ranges.push_back(Range{p, count, op.kind, op.delta, op.dst, op.own, op.dst2, op.own2, op.src});
    }
  }
  if (!l.ranges.empty()) out->push_back(l);
}

}  // namespace

// Ring of Sec. 6: 2(P - 1) single-placement launches, all in place.
static void ring_launches(Schedule* s) {
  const int32_t P = s->P;
  for (int32_t i = 0; i + 1 < P; ++i) {
    std::vector<std::vector<POp>> per_p(P);
    per_p[i + 1].push_back(POp{kReduce, -1, kBufU, kBufU, kBufNone, kBufNone, kBufU});
    emit_launch(&s->launches, kPhaseReduce, per_p);
  }
  for (int32_t j = 0; j + 1 < P; ++j) {
    std::vector<std::vector<POp>> per_p(P);
    per_p[j].push_back(POp{kCopy, -1, kBufU, kBufNone, kBufNone, kBufNone, kBufU});
    emit_launch(&s->launches, kPhaseDistribute, per_p);
  }
  s->rs_steps = P - 1;
  s->ag_steps = P - 1;
}

// Butterfly schedules over the XOR group (power-of-two P).
static void xor_launches(Schedule* s) {
  const int32_t P = s->P, L = s->L, r = s->r, w = s->w;
  // buffer written by reduction step i: U in place while f_i >= w (but X for
  // the last such step when a single doubling step follows, which must not
  // read and write U at once), then X / Y alternating so that the last step
  // writes U.
  auto rd_dst = [&](int32_t i) {
    const int32_t back = L - 1 - i;
    return back == 0 ? kBufU : (back % 2 == 1 ? kBufX : kBufY);
  };
  int32_t prim = kBufU;
  bool local_copy = false;
  for (int32_t i = 0; i < L; ++i) {
    const int32_t f = P >> (i + 1);
    std::vector<std::vector<POp>> per_p(P);
    if (f >= w) {
      const int32_t dst = (r == 1 && f == w) ? kBufX : kBufU;
      for (int32_t p = 0; p < f; ++p) per_p[p].push_back(POp{kReduce, f, dst, kBufU, kBufNone, kBufNone, kBufU});
      prim = dst;
    } else {
      int32_t dst = rd_dst(i);
      if (dst == prim) {  // P = 2, k = 1: the only step reads U
        dst = kBufX;
        local_copy = true;
      }
      for (int32_t p = 0; p < w; ++p) per_p[p].push_back(POp{kReduce, f, dst, prim, kBufNone, kBufNone, prim});
      prim = dst;
    }
    if (prim != kBufU) s->uses_scratch = true;
    emit_launch(&s->launches, kPhaseReduce, per_p);
  }
  if (local_copy) {
    std::vector<std::vector<POp>> cp_p(P);
    for (int32_t p = 0; p < w; ++p) cp_p[p].push_back(POp{kCopy, 0, kBufU, kBufNone, kBufNone, kBufNone, kBufX});
    emit_launch(&s->launches, kPhaseLocal, cp_p);
  }
  s->rs_steps = L;
  for (int32_t i = L - 1; i >= 0; --i) {
    const int32_t f = P >> (i + 1);
    if (2 * f <= w) continue;
    std::vector<std::vector<POp>> per_p(P);
    for (int32_t p = f; p < 2 * f; ++p) per_p[p].push_back(POp{kCopy, f, kBufU, kBufNone, kBufNone, kBufNone, kBufU});
    emit_launch(&s->launches, kPhaseDistribute, per_p);
    ++s->ag_steps;
  }
}

std::string build_schedule(int32_t P, int64_t n, int32_t k, Schedule* out) {
  return build_schedule_ex(P, n, k, kGroupCyclic, kSchedButterfly, out);
}

std::string build_schedule_ex(int32_t P, int64_t n, int32_t k, int32_t group, int32_t sched, Schedule* out) {
  Schedule s;
  if (P < 1 || P > kMaxP) return "P must be in [1, 128]";
  if (n < 0 || n > kMaxRankElems) return "n must be in [0, 2^46]";
  if (group != kGroupCyclic && group != kGroupXor) return "unknown group";
  if (sched != kSchedButterfly && sched != kSchedRing) return "unknown schedule";
  if (group == kGroupXor && (P & (P - 1)) != 0) return "the XOR group needs a power-of-two P";
  if (sched == kSchedRing && group != kGroupCyclic) return "the Ring schedule runs over the cyclic group";
  s.P = P;
  s.n = n;
  s.L = ceil_log2(P);
  s.group = group;
  s.sched = sched;
  if (sched == kSchedRing) {
    if (k != 2 * (P - 1)) {
      char buf[96];
      std::snprintf(buf, sizeof buf, "the Ring takes k_steps = 2(P-1) = %d for P=%d, got %d", 2 * (P - 1), P, k);
      return buf;
    }
  } else if (k < s.L || k > 2 * s.L) {
    char buf[96];
    std::snprintf(buf, sizeof buf, "k_steps=%d outside [%d, %d] for P=%d", k, s.L, 2 * s.L, P);
    return buf;
  }
  s.k = k;
  s.r = sched == kSchedRing ? 0 : 2 * s.L - k;  // the Ring removes no distribution step
  s.w = int32_t(std::min<int64_t>(int64_t(1) << s.r, P));
  s.N.assign(s.L + 1, 0);
  s.f.assign(s.L, 0);
  s.c.assign(s.L, 0);
  s.N[0] = P;
  for (int32_t i = 0; i < s.L; ++i) {
    s.f[i] = s.N[i] / 2;
    s.c[i] = s.N[i] - s.f[i];
    s.N[i + 1] = s.c[i];
  }

  const int32_t w = s.w;
  auto in_S = [&](int32_t p) { return p < w; };

  if (sched == kSchedRing) {
    ring_launches(&s);
  } else if (group == kGroupXor) {
    xor_launches(&s);
  } else {
  // ---- reduction phase ----
  if (s.r == 0) {
    for (int32_t i = 0; i < s.L; ++i) {
      std::vector<std::vector<POp>> per_p(P);
      for (int32_t p = s.c[i] - s.f[i]; p < s.c[i]; ++p)
        per_p[p].push_back(POp{kReduce, s.f[i], kBufU, kBufU, kBufNone, kBufNone, kBufU});
      emit_launch(&s.launches, kPhaseReduce, per_p);
    }
  } else {
    s.uses_scratch = true;
    int32_t prim = kBufU;  // buffer holding the primed sums read in this step
    bool aliased = true;   // starred sums still equal the primed ones
    for (int32_t i = 0; i < s.L; ++i) {
      const int32_t f = s.f[i], c = s.c[i], N = s.N[i];
      const bool even = (N % 2) == 0, last = (i == s.L - 1);
      const int32_t next = (i % 2 == 0) ? kBufX : kBufY;
      // primed placements still needed afterwards: S + [1, c)
      const int32_t cp = c >= 2 ? std::min(P, w + c - 2) : 0;
      auto in_PO = [&](int32_t p) { return cp > 0 && pmod(p - 1, P) < cp; };
      std::vector<std::vector<POp>> per_p(P);
      bool local_copy = false;
      for (int32_t p = 0; p < P; ++p) {
        if (aliased) {
          if (even && !last) {
            if (in_S(p) || in_PO(p)) per_p[p].push_back(POp{kReduce, f, next, prim, kBufNone, kBufNone, prim});
          } else if (even && last) {
            if (in_S(p)) {
              const int32_t dst = prim == kBufU ? next : kBufU;  // P = 2, k = 1 reads and writes U
              local_copy = prim == kBufU;
              per_p[p].push_back(POp{kReduce, f, dst, prim, kBufNone, kBufNone, prim});
            }
          } else {  // odd step: starred sums stop following the primed ones
            if (in_PO(p)) per_p[p].push_back(POp{kReduce, f, next, prim, kBufNone, kBufNone, prim});
            if (in_S(p) && prim != kBufU)
              per_p[p].push_back(POp{kCopy, 0, kBufU, kBufNone, kBufNone, kBufNone, prim});
          }
        } else {
          const bool po = in_PO(p), st = in_S(p) && even;
          if (po && st)
            per_p[p].push_back(POp{kReduce2, f, next, prim, kBufU, kBufU, prim});
          else if (po)
            per_p[p].push_back(POp{kReduce, f, next, prim, kBufNone, kBufNone, prim});
          else if (st)
            per_p[p].push_back(POp{kReduce, f, kBufU, kBufU, kBufNone, kBufNone, prim});
        }
      }
      emit_launch(&s.launches, kPhaseReduce, per_p);
      if (local_copy) {
        std::vector<std::vector<POp>> cp_p(P);
        for (int32_t p = 0; p < w; ++p) cp_p[p].push_back(POp{kCopy, 0, kBufU, kBufNone, kBufNone, kBufNone, next});
        emit_launch(&s.launches, kPhaseLocal, cp_p);
      }
      if (aliased && !even) aliased = false;
      prim = next;
    }
  }
  s.rs_steps = s.L;

  // ---- distribution phase ----
  int32_t h = w;
  for (int32_t i = s.L - 1; i >= 0; --i) {
    if (s.N[i] <= h) continue;
    const int32_t lo = std::max(s.c[i], h);
    std::vector<std::vector<POp>> per_p(P);
    for (int32_t p = lo; p < s.N[i]; ++p)
      per_p[p].push_back(POp{kCopy, -s.f[i], kBufU, kBufNone, kBufNone, kBufNone, kBufU});
    emit_launch(&s.launches, kPhaseDistribute, per_p);
    ++s.ag_steps;
    h = s.N[i];
  }
  }  // cyclic butterfly

  // ---- sizes ----
  for (const Launch& l : s.launches) {
    std::set<std::pair<int32_t, int32_t>> pulled;  // (src buffer, source placement)
    for (const Range& rg : l.ranges) {
      for (int32_t j = 0; j < rg.count; ++j) {
        const int32_t p = pmod(rg.p0 + j, P);
        if (rg.delta != 0) pulled.insert({rg.src, group == kGroupXor ? (p ^ rg.delta) : pmod(p + rg.delta, P)});
        s.combines_per_rank += rg.kind == kReduce ? 1 : rg.kind == kReduce2 ? 2 : 0;
        s.hbm_blocks += rg.kind == kCopy ? 2 : rg.kind == kReduce ? 3 : 5;
      }
    }
    s.blocks_pulled_per_rank += int64_t(pulled.size());
  }
  for (const Launch& l : s.launches)
    for (const Range& rg : l.ranges)
      if (rg.count < 1 || rg.count > P) return "internal: empty or oversized range";
  for (const Launch& l : s.launches)
    if (int32_t(l.ranges.size()) > kMaxRanges) return "internal: too many placement ranges in one launch";

  std::string hz = check_hazards(s);
  if (!hz.empty()) return "internal: " + hz;
  *out = std::move(s);
  return "";
}

// Every work item is (rank x, range, placement p).  A location is (buffer,
// rank, block).  Inside one launch no location may be written by one item and
// read or written by another; an item may read and write its own location
// (in-place combination).
std::string check_hazards(const Schedule& s) {
  const int32_t P = s.P;
  auto key = [P](int32_t buf, int32_t rank, int32_t blk) { return (int64_t(buf) * P + rank) * P + blk; };
  std::vector<int64_t> writer(size_t(3) * P * P);
  for (size_t li = 0; li < s.launches.size(); ++li) {
    const Launch& l = s.launches[li];
    std::fill(writer.begin(), writer.end(), -1);
    int64_t item = 0;
    // writes
    for (const Range& rg : l.ranges)
      for (int32_t j = 0; j < rg.count; ++j)
        for (int32_t x = 0; x < P; ++x, ++item) {
          const int32_t p = pmod(rg.p0 + j, P), b = group_block(s.group, x, p, P);
          for (int32_t d : {rg.dst, rg.dst2}) {
            if (d == kBufNone) continue;
            int64_t& wv = writer[key(d, x, b)];
            if (wv >= 0) return "launch " + std::to_string(li) + ": two writers of one block";
            wv = item;
          }
        }
    // reads
    item = 0;
    for (const Range& rg : l.ranges)
      for (int32_t j = 0; j < rg.count; ++j)
        for (int32_t x = 0; x < P; ++x, ++item) {
          const int32_t p = pmod(rg.p0 + j, P), b = group_block(s.group, x, p, P);
          const int32_t y = group_peer(s.group, x, rg.delta, P);
          const int64_t reads[3] = {rg.own == kBufNone ? -1 : key(rg.own, x, b),
                                    rg.own2 == kBufNone ? -1 : key(rg.own2, x, b),
                                    rg.src == kBufNone ? -1 : key(rg.src, y, b)};
          for (int64_t rk : reads) {
            if (rk < 0) continue;
            if (writer[rk] >= 0 && writer[rk] != item)
              return "launch " + std::to_string(li) + ": a block read by one rank is written by another";
          }
        }
  }
  return "";
}

}  // namespace ar
