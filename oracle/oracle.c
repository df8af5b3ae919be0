/*
 * oracle.c -- plain, slow CPU reference for the generalized Allreduce of
 * Kolmakov & Zhang, "A Generalization of the Allreduce Operation"
 * (arXiv:2004.09362).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  It shares no code, header,
 * table or constant with the HIP library it checks, and the HIP library never
 * calls it.
 *
 * What it computes
 * ----------------
 *  1. oracle_direct_*: the plain definition of Allreduce -- every rank ends
 *     with the elementwise combination of all P input vectors (Sec. 1, the
 *     definition of the operation; Sec. 5.4, the per-element reduction
 *     result u_{i,Sigma}).  int32 sums wrap modulo 2^32; fp32 sums are
 *     accumulated in fp64.
 *  2. oracle_allreduce: a rank-by-rank replay of the paper's schedule in the
 *     input precision, following the paper's steps in its own order:
 *       - cyclic group T_P with generator x -> x+1 (Sec. 5), placement
 *         permutation h = identity, so the distributed vector t^p q holds
 *         block (x - p) mod P on rank x (Sec. 5.1, 5.2);
 *       - reduction phase of the bandwidth-optimal algorithm (Sec. 7):
 *         N_0 = P, N_{i+1} = ceil(N_i / 2), operator t^{-floor(N_i/2)}
 *         applied to the vectors [ceil(N_i/2), N_i) of the current set, each
 *         received vector combined with the co-placed kept one (eqs. for the
 *         starting set, its size, the step operator, the sent set and the
 *         even/odd step results);
 *       - the schedule shifted by s = 0 .. w-1 with unchanged operators, so
 *         that the reduction ends holding t^0 q_Sigma .. t^{w-1} q_Sigma and
 *         the first r distribution steps disappear (Sec. 8, the shifted
 *         starting set); w = min(2^r, P), r = 2*ceil(log2 P) - k; r equal to
 *         ceil(log2 P) is the latency-optimal corner case (Sec. 9);
 *       - distribution phase: the reduction steps reversed, without
 *         combination (Sec. 7, the paragraph after the last-step equation;
 *         Sec. 6, the inverse operators), fetching only placements that are
 *         not held yet.
 *     Every shift is simulated as its own independent schedule.  Within a
 *     step all ranks send first (into per-rank receive buffers) and combine
 *     afterwards, i.e. the exchange is simultaneous (Sec. 5.3).
 *     The same replay runs over the group of Sec. 4's Table 1b for
 *     power-of-two P -- t_k(x) = x XOR k, every element self-inverse -- in
 *     which the bandwidth-optimal schedule is Recursive Halving and the
 *     latency-optimal one Recursive Doubling (Secs. 7 and 8, closing
 *     remarks).  Group arithmetic is written through grp_mul / grp_inv:
 *     placement of vector v of shift s is s.v, rank x holds block x.p^-1 of
 *     placement p, a reduction step with operator t_f^-1 brings rank x the
 *     vectors of rank x.f, and vector v lands as f^-1.v.
 *  2b. oracle_allreduce_ex with the Ring schedule of Sec. 6: over the cyclic
 *     group with the operator t at every step, P - 1 reduction steps (rank
 *     x receives the partial sum of rank x - 1, placement i, and combines it
 *     with its own placement i + 1) and P - 1 distribution steps with the
 *     same operator.
 *  3. A symbolic "term" mode of the same replay: values are nodes of a
 *     hash-consed expression DAG, so the reduction tree of every output can
 *     be printed and compared with the paper's worked P = 7 example, every
 *     combine can be checked to join disjoint sets of ranks of one block,
 *     and the number of distinct vectors sent / combined per step can be
 *     counted against the cost equations of Secs. 7-9.
 *
 * Readings taken where the paper is silent (each one is listed with its
 * reason in the design notes of the repository):
 *   - block sizes when P does not divide n: the first (n mod P) blocks hold
 *     ceil(n/P) elements, the others floor(n/P);
 *   - combination operand order: kept (own) vector first, received second;
 *   - max: (recv > own) ? recv : own;
 *   - shifts for r > 1: s = 0 .. 2^r - 1, clipped to P;
 *   - distribution after a shifted reduction fetches placements
 *     [max(ceil(N_i/2), h), N_i) where [0, h) are already held.
 *
 * Parity pinning: see tests/test_oracle_pins.py.  The fp32-sum replay bits
 * are pinned only through the paper's worked P = 7 and P = 3 trees and the
 * tree-shape checks of the term mode; elsewhere fp32 sums are held to an
 * error bound against the fp64 direct sum.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#define ORC_MAXP 128
#define ORC_MAX_STEPS 16

enum { ORC_I32_SUM = 0, ORC_I32_MAX = 1, ORC_F32_SUM = 2, ORC_F32_MAX = 3, ORC_TERM = 4 };
enum { ORC_GROUP_CYCLIC = 0, ORC_GROUP_XOR = 1 };
enum { ORC_SCHED_BUTTERFLY = 0, ORC_SCHED_RING = 1 };

/* ------------------------------------------------------------------------ */
/* Term DAG (symbolic mode)                                                  */
/* ------------------------------------------------------------------------ */

typedef struct orc_terms {
  int32_t P;          /* leaves are ids [0, P*P): leaf(y, b) = y*P + b      */
  int64_t n_nodes;    /* total ids in use (leaves included)                 */
  int64_t cap;
  int32_t* left;      /* per id; -1 for a leaf                              */
  int32_t* right;
  int32_t* blk;       /* block the value belongs to                         */
  uint64_t* mask;     /* two words per id: set of source ranks              */
  int64_t hcap;       /* hash table of (left,right) -> id                   */
  int32_t* htab;
  int64_t violations; /* combines of overlapping sets or of different blocks*/
} orc_terms;

orc_terms* oracle_terms_new(void) {
  orc_terms* t = (orc_terms*)calloc(1, sizeof(orc_terms));
  return t;
}

void oracle_terms_free(orc_terms* t) {
  if (!t) return;
  free(t->left); free(t->right); free(t->blk); free(t->mask); free(t->htab);
  free(t);
}

static int terms_grow(orc_terms* t, int64_t need) {
  if (need <= t->cap) return 0;
  int64_t nc = t->cap ? t->cap : 1024;
  while (nc < need) nc *= 2;
  int32_t* l = (int32_t*)realloc(t->left, nc * sizeof(int32_t));
  if (!l) return -1;
  t->left = l;
  int32_t* r = (int32_t*)realloc(t->right, nc * sizeof(int32_t));
  if (!r) return -1;
  t->right = r;
  int32_t* b = (int32_t*)realloc(t->blk, nc * sizeof(int32_t));
  if (!b) return -1;
  t->blk = b;
  uint64_t* m = (uint64_t*)realloc(t->mask, nc * 2 * sizeof(uint64_t));
  if (!m) return -1;
  t->mask = m;
  t->cap = nc;
  return 0;
}

static uint64_t pair_hash(int32_t a, int32_t b) {
  uint64_t h = ((uint64_t)(uint32_t)a << 32) | (uint32_t)b;
  h ^= h >> 33; h *= 0xff51afd7ed558ccdULL; h ^= h >> 33; h *= 0xc4ceb9fe1a85ec53ULL; h ^= h >> 33;
  return h;
}

static int terms_rehash(orc_terms* t, int64_t ncap) {
  int32_t* nt = (int32_t*)malloc(ncap * sizeof(int32_t));
  if (!nt) return -1;
  for (int64_t i = 0; i < ncap; ++i) nt[i] = -1;
  for (int64_t id = (int64_t)t->P * t->P; id < t->n_nodes; ++id) {
    uint64_t h = pair_hash(t->left[id], t->right[id]) & (uint64_t)(ncap - 1);
    while (nt[h] >= 0) h = (h + 1) & (uint64_t)(ncap - 1);
    nt[h] = (int32_t)id;
  }
  free(t->htab);
  t->htab = nt;
  t->hcap = ncap;
  return 0;
}

/* Reset the DAG for P ranks and create the P*P leaves. */
static int terms_reset(orc_terms* t, int32_t P) {
  t->P = P;
  t->n_nodes = 0;
  t->violations = 0;
  if (terms_grow(t, (int64_t)P * P + 16)) return -1;
  for (int32_t y = 0; y < P; ++y)
    for (int32_t b = 0; b < P; ++b) {
      int64_t id = (int64_t)y * P + b;
      t->left[id] = -1;
      t->right[id] = -1;
      t->blk[id] = b;
      t->mask[2 * id] = y < 64 ? (1ULL << y) : 0;
      t->mask[2 * id + 1] = y >= 64 ? (1ULL << (y - 64)) : 0;
    }
  t->n_nodes = (int64_t)P * P;
  return terms_rehash(t, 1024);
}

/* own (+) recv as a DAG node; identical sub-trees get identical ids. */
static int32_t terms_combine(orc_terms* t, int32_t a, int32_t b) {
  if (t->blk[a] != t->blk[b]) t->violations++;
  if ((t->mask[2 * a] & t->mask[2 * b]) || (t->mask[2 * a + 1] & t->mask[2 * b + 1])) t->violations++;
  uint64_t h = pair_hash(a, b) & (uint64_t)(t->hcap - 1);
  while (t->htab[h] >= 0) {
    int32_t id = t->htab[h];
    if (t->left[id] == a && t->right[id] == b) return id;
    h = (h + 1) & (uint64_t)(t->hcap - 1);
  }
  if (terms_grow(t, t->n_nodes + 1)) return -1;
  int64_t id = t->n_nodes++;
  t->left[id] = a;
  t->right[id] = b;
  t->blk[id] = t->blk[a];
  t->mask[2 * id] = t->mask[2 * a] | t->mask[2 * b];
  t->mask[2 * id + 1] = t->mask[2 * a + 1] | t->mask[2 * b + 1];
  t->htab[h] = (int32_t)id;
  if (2 * (t->n_nodes - (int64_t)t->P * t->P) > t->hcap) {
    if (terms_rehash(t, t->hcap * 2)) return -1;
  }
  return (int32_t)id;
}

int64_t oracle_terms_violations(const orc_terms* t) { return t->violations; }
int64_t oracle_terms_count(const orc_terms* t) { return t->n_nodes; }

void oracle_terms_mask(const orc_terms* t, int32_t id, uint64_t* out2) {
  out2[0] = t->mask[2 * id];
  out2[1] = t->mask[2 * id + 1];
}

int32_t oracle_terms_block(const orc_terms* t, int32_t id) { return t->blk[id]; }

/* Render a node as text: a leaf is the source rank number, a combine is
 * "(own+recv)".  Returns the length written, or -1 if cap is too small. */
static int64_t render_rec(const orc_terms* t, int32_t id, char* buf, int64_t cap, int64_t pos) {
  if (pos < 0) return -1;
  if (t->left[id] < 0) {
    int32_t y = id / t->P;
    int w = snprintf(buf + pos, (size_t)(cap > pos ? cap - pos : 0), "%d", y);
    if (w < 0 || pos + w >= cap) return -1;
    return pos + w;
  }
  if (pos + 1 >= cap) return -1;
  buf[pos++] = '(';
  pos = render_rec(t, t->left[id], buf, cap, pos);
  if (pos < 0 || pos + 1 >= cap) return -1;
  buf[pos++] = '+';
  pos = render_rec(t, t->right[id], buf, cap, pos);
  if (pos < 0 || pos + 1 >= cap) return -1;
  buf[pos++] = ')';
  buf[pos] = 0;
  return pos;
}

int64_t oracle_terms_render(const orc_terms* t, int32_t id, char* buf, int64_t cap) {
  if (cap < 2) return -1;
  buf[0] = 0;
  return render_rec(t, id, buf, cap, 0);
}

/* ------------------------------------------------------------------------ */
/* Schedule parameters                                                       */
/* ------------------------------------------------------------------------ */

typedef struct {
  int32_t P, L, k, r, w;
  int32_t N[ORC_MAX_STEPS + 1], f[ORC_MAX_STEPS], c[ORC_MAX_STEPS];
} sched_t;

static int32_t ceil_log2_i(int32_t P) {
  int32_t L = 0;
  while ((1 << L) < P) ++L;
  return L;
}

/* Returns 0 on success, -1 for an unsupported (P, k). */
static int sched_init(sched_t* s, int32_t P, int32_t k) {
  if (P < 1 || P > ORC_MAXP) return -1;
  s->P = P;
  s->L = ceil_log2_i(P);
  if (k < s->L || k > 2 * s->L) return -1;
  s->k = k;
  s->r = 2 * s->L - k;                      /* distribution steps removed */
  s->w = (1 << s->r) < P ? (1 << s->r) : P; /* shifted schedules         */
  s->N[0] = P;
  for (int32_t i = 0; i < s->L; ++i) {
    s->f[i] = s->N[i] / 2;                  /* operator t^{-floor(N_i/2)} */
    s->c[i] = s->N[i] - s->f[i];            /* ceil(N_i / 2)              */
    s->N[i + 1] = s->c[i];
  }
  return 0;
}

/* Balanced block partition of n elements into P blocks: block b starts at
 * b*floor(n/P) + min(b, n mod P); this returns the block of element e. */
static int32_t blk_of(int64_t n, int32_t P, int64_t e) {
  int64_t q = n / P, m = n % P;
  if (e < m * (q + 1)) return (int32_t)(e / (q + 1));
  return (int32_t)(m + (e - m * (q + 1)) / q);
}

static int32_t mod_p(int64_t a, int32_t P) {
  int64_t v = a % P;
  return (int32_t)(v < 0 ? v + P : v);
}

/* Product and inverse in the group T_P acting on {0..P-1}: the cyclic group
 * (t_a t_b = t_{a+b mod P}) or the group of Table 1b (t_a t_b = t_{a XOR b},
 * P a power of two). */
static int32_t grp_mul(int32_t g, int32_t a, int32_t b, int32_t P) {
  return g == ORC_GROUP_XOR ? (a ^ b) : mod_p((int64_t)a + b, P);
}

static int32_t grp_inv(int32_t g, int32_t a, int32_t P) {
  return g == ORC_GROUP_XOR ? a : mod_p(-(int64_t)a, P);
}

/* ------------------------------------------------------------------------ */
/* Elementwise combination of two co-placed blocks (Sec. 5.4)                */
/* ------------------------------------------------------------------------ */

static int combine_block(int32_t kind, orc_terms* terms, void* dst, const void* own, const void* recv,
                         int64_t len) {
  int64_t e;
  switch (kind) {
    case ORC_I32_SUM: {
      const uint32_t* a = (const uint32_t*)own; const uint32_t* b = (const uint32_t*)recv;
      uint32_t* d = (uint32_t*)dst;
      for (e = 0; e < len; ++e) d[e] = a[e] + b[e];   /* wraps modulo 2^32 */
      return 0;
    }
    case ORC_I32_MAX: {
      const int32_t* a = (const int32_t*)own; const int32_t* b = (const int32_t*)recv;
      int32_t* d = (int32_t*)dst;
      for (e = 0; e < len; ++e) d[e] = b[e] > a[e] ? b[e] : a[e];
      return 0;
    }
    case ORC_F32_SUM: {
      const float* a = (const float*)own; const float* b = (const float*)recv;
      float* d = (float*)dst;
      for (e = 0; e < len; ++e) d[e] = a[e] + b[e];
      return 0;
    }
    case ORC_F32_MAX: {
      const float* a = (const float*)own; const float* b = (const float*)recv;
      float* d = (float*)dst;
      for (e = 0; e < len; ++e) d[e] = b[e] > a[e] ? b[e] : a[e];
      return 0;
    }
    case ORC_TERM: {
      const int32_t* a = (const int32_t*)own; const int32_t* b = (const int32_t*)recv;
      int32_t* d = (int32_t*)dst;
      for (e = 0; e < len; ++e) {
        int32_t id = terms_combine(terms, a[e], b[e]);
        if (id < 0) return -1;
        d[e] = id;
      }
      return 0;
    }
  }
  return -1;
}

/* ------------------------------------------------------------------------ */
/* Trace of the schedule (sizes of what was sent and combined)               */
/* ------------------------------------------------------------------------ */

typedef struct {
  int32_t P, L, k, r, w;
  int32_t rs_steps, ag_steps;
  int32_t step_peer[ORC_MAX_STEPS];   /* receive from rank x.step_peer (group
                                         product; -1: from rank x - 1, Ring) */
  int32_t pulls[ORC_MAX_STEPS];       /* distinct vectors received, rank 0  */
  int32_t combines[ORC_MAX_STEPS];    /* distinct combine results, rank 0   */
  /* per step and rank: bitmask of the blocks received in that step */
  uint64_t recv_blocks[ORC_MAX_STEPS][ORC_MAXP][2];
} oracle_trace;

static void mark_block(oracle_trace* tr, int32_t step, int32_t x, int32_t b) {
  if (!tr) return;
  tr->recv_blocks[step][x][b >> 6] |= 1ULL << (b & 63);
}

/* A small set of int32 ids (distinct counting for the trace). */
typedef struct { int32_t* v; int64_t n, cap; } idset_t;

static int idset_add(idset_t* s, int32_t id) {
  for (int64_t i = 0; i < s->n; ++i) if (s->v[i] == id) return 0;
  if (s->n == s->cap) {
    int64_t nc = s->cap ? 2 * s->cap : 64;
    int32_t* nv = (int32_t*)realloc(s->v, nc * sizeof(int32_t));
    if (!nv) return -1;
    s->v = nv; s->cap = nc;
  }
  s->v[s->n++] = id;
  return 0;
}

/* ------------------------------------------------------------------------ */
/* The schedule replay                                                       */
/* ------------------------------------------------------------------------ */

/*
 * oracle_allreduce -- replay the schedule for (P, k) on rank data.
 *
 *   in   : element (y, j) at in  + (y * in_rank_stride  + j) * 4 bytes, the
 *          value of rank y at global column cols[j] (cols[j] = j if cols is
 *          NULL, then ncols must equal n).  4-byte elements: int32, float or,
 *          in term mode, ignored on input.
 *   out  : same layout with out_rank_stride; receives every rank's result.
 *   cols : strictly increasing global column indices in [0, n): the replay
 *          of a column depends only on the block the column falls in, so a
 *          sample of columns gives exactly the values the full run gives at
 *          those columns.
 *   terms: required in term mode (kind ORC_TERM); leaves are leaf(y, b).
 *   trace: optional; filled with the step sizes.
 * Returns 0, or -1 for bad arguments / allocation failure.
 */
static int ring_replay(int32_t P, int64_t n, int32_t k, int32_t kind, const void* in, int64_t in_rank_stride,
                       void* out, int64_t out_rank_stride, const int64_t* cols, int64_t ncols, orc_terms* terms,
                       oracle_trace* trace);

int oracle_allreduce_ex(int32_t P, int64_t n, int32_t k, int32_t kind, int32_t group, int32_t schedule,
                        const void* in, int64_t in_rank_stride,
                        void* out, int64_t out_rank_stride,
                        const int64_t* cols, int64_t ncols,
                        orc_terms* terms, oracle_trace* trace) {
  if (group != ORC_GROUP_CYCLIC && group != ORC_GROUP_XOR) return -1;
  if (group == ORC_GROUP_XOR && (P & (P - 1)) != 0) return -1;   /* needs a power of two */
  if (schedule == ORC_SCHED_RING) {
    if (group != ORC_GROUP_CYCLIC) return -1;
    return ring_replay(P, n, k, kind, in, in_rank_stride, out, out_rank_stride, cols, ncols, terms, trace);
  }
  if (schedule != ORC_SCHED_BUTTERFLY) return -1;
  const int32_t g = group;
  sched_t s;
  if (sched_init(&s, P, k)) return -1;
  if (n < 0 || ncols < 0 || (!cols && ncols != n)) return -1;
  if (kind < 0 || kind > ORC_TERM) return -1;
  if (kind == ORC_TERM && !terms) return -1;
  if (kind == ORC_TERM && terms_reset(terms, P)) return -1;
  for (int64_t j = 0; j < ncols; ++j) {
    int64_t e = cols ? cols[j] : j;
    if (e < 0 || e >= n || (j > 0 && cols && cols[j] <= cols[j - 1])) return -1;
  }

  /* Columns of each block: a contiguous range [gs[b], gs[b+1]) of j. */
  int64_t gs[ORC_MAXP + 1];
  {
    int32_t b = 0;
    gs[0] = 0;
    for (int64_t j = 0; j < ncols; ++j) {
      int32_t bj = blk_of(n, P, cols ? cols[j] : j);
      while (b < bj) gs[++b] = j;
    }
    while (b < P) gs[++b] = ncols;
  }

  const int64_t ES = 4; /* element size */
  int64_t cells = (int64_t)P * ncols;
  char* W = (char*)malloc((size_t)(cells ? cells : 1) * ES);    /* vectors of one shift  */
  char* M = (char*)malloc((size_t)(cells ? cells : 1) * ES);    /* per-rank receive area  */
  char* F = (char*)malloc((size_t)(cells ? cells : 1) * ES);    /* final placements       */
  if (!W || !M || !F) { free(W); free(M); free(F); return -1; }
#define CELL(buf, x, j) ((buf) + ((int64_t)(x) * ncols + (j)) * ES)

  idset_t recv_ids[ORC_MAX_STEPS], comb_ids[ORC_MAX_STEPS];
  memset(recv_ids, 0, sizeof(recv_ids));
  memset(comb_ids, 0, sizeof(comb_ids));
  if (trace) {
    memset(trace, 0, sizeof(*trace));
    trace->P = P; trace->L = s.L; trace->k = k; trace->r = s.r; trace->w = s.w;
    trace->rs_steps = s.L;
  }
  int rc = 0;

  /* ---- reduction phase: one independent schedule per shift s ---- */
  for (int32_t sh = 0; sh < s.w && rc == 0; ++sh) {
    /* Initial set of distributed vectors: every rank holds its own data. */
    for (int32_t x = 0; x < P; ++x)
      for (int64_t j = 0; j < ncols; ++j) {
        if (kind == ORC_TERM) {
          int32_t id = x * P + blk_of(n, P, cols ? cols[j] : j);
          memcpy(CELL(W, x, j), &id, 4);
        } else {
          memcpy(CELL(W, x, j), (const char*)in + ((int64_t)x * in_rank_stride + j) * ES, ES);
        }
      }
    for (int32_t i = 0; i < s.L && rc == 0; ++i) {
      const int32_t f = s.f[i], c = s.c[i], N = s.N[i];
      if (trace) trace->step_peer[i] = f;
      /* Send: with operator t_f^-1 rank y sends its blocks of vectors v in
       * [c, N) of this shift to rank f^-1.y; rank x therefore receives from
       * x.f the block of vector v, which on x.f is block (x.f).(sh.v)^-1. */
      for (int32_t x = 0; x < P; ++x) {
        int32_t y = grp_mul(g, x, f, P);
        for (int32_t v = c; v < N; ++v) {
          int32_t b = grp_mul(g, y, grp_inv(g, grp_mul(g, sh, v, P), P), P);
          for (int64_t j = gs[b]; j < gs[b + 1]; ++j) memcpy(CELL(M, x, j), CELL(W, y, j), ES);
          if (trace) mark_block(trace, i, x, b);
          if (trace && x == 0 && kind == ORC_TERM && gs[b + 1] > gs[b]) {
            int32_t id; memcpy(&id, CELL(W, y, gs[b]), 4);
            if (idset_add(&recv_ids[i], id)) rc = -1;
          }
        }
      }
      /* Combine: the received vector v now sits where vector f^-1.v of the
       * shift is kept (v - f, or v XOR f), co-placed with it; own value
       * first, received second. */
      for (int32_t x = 0; x < P && rc == 0; ++x) {
        for (int32_t v = c; v < N; ++v) {
          int32_t kept = grp_mul(g, grp_inv(g, f, P), v, P);
          int32_t b = grp_mul(g, x, grp_inv(g, grp_mul(g, sh, kept, P), P), P);
          int64_t j0 = gs[b], len = gs[b + 1] - gs[b];
          if (len == 0) continue;
          if (combine_block(kind, terms, CELL(W, x, j0), CELL(W, x, j0), CELL(M, x, j0), len)) { rc = -1; break; }
          if (trace && x == 0 && kind == ORC_TERM) {
            int32_t id; memcpy(&id, CELL(W, x, j0), 4);
            if (idset_add(&comb_ids[i], id)) rc = -1;
          }
        }
      }
    }
    /* After the last step vector 0 of this shift (placement sh) holds the
     * complete result of block x.sh^-1 on every rank x. */
    for (int32_t x = 0; x < P; ++x) {
      int32_t b = grp_mul(g, x, grp_inv(g, sh, P), P);
      for (int64_t j = gs[b]; j < gs[b + 1]; ++j) memcpy(CELL(F, x, j), CELL(W, x, j), ES);
    }
  }

  /* ---- distribution phase: reduction steps reversed, no combination ---- */
  int32_t h = s.w;            /* placements [0, h) are held on every rank */
  int32_t step = s.L;
  for (int32_t i = s.L - 1; i >= 0 && rc == 0; --i) {
    if (s.N[i] <= h) continue;     /* omitted step: everything already held */
    const int32_t f = s.f[i];
    const int32_t lo = s.c[i] > h ? s.c[i] : h;
    if (trace) trace->step_peer[step] = -f;
    /* Operator t_f: placement f^-1.p of rank x.f^-1 moves to placement p of
     * rank x (same block).  Receive everything first, then store. */
    for (int32_t x = 0; x < P; ++x) {
      int32_t y = grp_mul(g, x, grp_inv(g, f, P), P);
      for (int32_t p = lo; p < s.N[i]; ++p) {
        int32_t b = grp_mul(g, x, grp_inv(g, p, P), P);
        for (int64_t j = gs[b]; j < gs[b + 1]; ++j) memcpy(CELL(M, x, j), CELL(F, y, j), ES);
        if (trace) mark_block(trace, step, x, b);
      }
    }
    for (int32_t x = 0; x < P; ++x)
      for (int32_t p = lo; p < s.N[i]; ++p) {
        int32_t b = grp_mul(g, x, grp_inv(g, p, P), P);
        for (int64_t j = gs[b]; j < gs[b + 1]; ++j) memcpy(CELL(F, x, j), CELL(M, x, j), ES);
      }
    if (trace) trace->pulls[step] = s.N[i] - lo;
    h = s.N[i];
    ++step;
  }
  if (trace) {
    trace->ag_steps = step - s.L;
    for (int32_t i = 0; i < s.L; ++i) {
      int32_t cnt = 0;
      for (int32_t b = 0; b < P; ++b) cnt += (int32_t)((trace->recv_blocks[i][0][b >> 6] >> (b & 63)) & 1);
      trace->pulls[i] = kind == ORC_TERM ? (int32_t)recv_ids[i].n : cnt;
      trace->combines[i] = kind == ORC_TERM ? (int32_t)comb_ids[i].n : -1;
    }
  }

  for (int32_t x = 0; x < P; ++x)
    for (int64_t j = 0; j < ncols; ++j)
      memcpy((char*)out + ((int64_t)x * out_rank_stride + j) * ES, CELL(F, x, j), ES);
#undef CELL
  for (int i = 0; i < ORC_MAX_STEPS; ++i) { free(recv_ids[i].v); free(comb_ids[i].v); }
  free(W); free(M); free(F);
  return rc;
}

/* The cyclic group and the butterfly schedules of Secs. 7-9. */
int oracle_allreduce(int32_t P, int64_t n, int32_t k, int32_t kind,
                     const void* in, int64_t in_rank_stride,
                     void* out, int64_t out_rank_stride,
                     const int64_t* cols, int64_t ncols,
                     orc_terms* terms, oracle_trace* trace) {
  return oracle_allreduce_ex(P, n, k, kind, ORC_GROUP_CYCLIC, ORC_SCHED_BUTTERFLY, in, in_rank_stride, out,
                             out_rank_stride, cols, ncols, terms, trace);
}

/*
 * Ring schedule of Sec. 6 (cyclic group, operator t every step), k = 2(P-1).
 * Placement p of rank x is block x - p.  Reduction step i = 0..P-2: the
 * partial sum at placement i of rank x - 1 moves to placement i + 1 of rank
 * x and is combined with rank x's own vector there (own first).  After
 * P - 1 steps placement P - 1 holds the full result of block x + 1; the
 * distribution steps j = 0..P-2 move placement j - 1 (mod P) of rank x - 1
 * to placement j of rank x.  Trace sizes are kept for at most
 * ORC_MAX_STEPS steps.
 */
static int ring_replay(int32_t P, int64_t n, int32_t k, int32_t kind, const void* in, int64_t in_rank_stride,
                       void* out, int64_t out_rank_stride, const int64_t* cols, int64_t ncols, orc_terms* terms,
                       oracle_trace* trace) {
  if (P < 1 || P > ORC_MAXP || k != 2 * (P - 1)) return -1;
  if (n < 0 || ncols < 0 || (!cols && ncols != n)) return -1;
  if (kind < 0 || kind > ORC_TERM) return -1;
  if (kind == ORC_TERM && !terms) return -1;
  if (kind == ORC_TERM && terms_reset(terms, P)) return -1;
  for (int64_t j = 0; j < ncols; ++j) {
    int64_t e = cols ? cols[j] : j;
    if (e < 0 || e >= n || (j > 0 && cols && cols[j] <= cols[j - 1])) return -1;
  }
  int64_t gs[ORC_MAXP + 1];
  {
    int32_t b = 0;
    gs[0] = 0;
    for (int64_t j = 0; j < ncols; ++j) {
      int32_t bj = blk_of(n, P, cols ? cols[j] : j);
      while (b < bj) gs[++b] = j;
    }
    while (b < P) gs[++b] = ncols;
  }
  const int64_t ES = 4;
  int64_t cells = (int64_t)P * ncols;
  char* W = (char*)malloc((size_t)(cells ? cells : 1) * ES);
  char* M = (char*)malloc((size_t)(cells ? cells : 1) * ES);
  if (!W || !M) { free(W); free(M); return -1; }
#define RCELL(buf, x, j) ((buf) + ((int64_t)(x) * ncols + (j)) * ES)
  for (int32_t x = 0; x < P; ++x)
    for (int64_t j = 0; j < ncols; ++j) {
      if (kind == ORC_TERM) {
        int32_t id = x * P + blk_of(n, P, cols ? cols[j] : j);
        memcpy(RCELL(W, x, j), &id, 4);
      } else {
        memcpy(RCELL(W, x, j), (const char*)in + ((int64_t)x * in_rank_stride + j) * ES, ES);
      }
    }
  if (trace) {
    memset(trace, 0, sizeof(*trace));
    trace->P = P; trace->k = k; trace->rs_steps = P - 1; trace->ag_steps = P - 1;
    trace->L = ceil_log2_i(P);
  }
  int rc = 0;
  for (int32_t step = 0; step < 2 * (P - 1) && rc == 0; ++step) {
    const int reduce = step < P - 1;
    const int32_t from_p = reduce ? step : mod_p((int64_t)step - P, P);
    const int32_t to_p = mod_p((int64_t)from_p + 1, P);
    /* receive: rank x gets rank x-1's placement from_p, block (x-1) - from_p */
    for (int32_t x = 0; x < P; ++x) {
      int32_t y = mod_p((int64_t)x - 1, P);
      int32_t b = mod_p((int64_t)y - from_p, P);
      for (int64_t j = gs[b]; j < gs[b + 1]; ++j) memcpy(RCELL(M, x, j), RCELL(W, y, j), ES);
      if (trace && step < ORC_MAX_STEPS) mark_block(trace, step, x, b);
    }
    /* combine (reduction) or store (distribution) at placement to_p */
    for (int32_t x = 0; x < P && rc == 0; ++x) {
      int32_t b = mod_p((int64_t)x - to_p, P);
      int64_t j0 = gs[b], len = gs[b + 1] - gs[b];
      if (len == 0) continue;
      if (reduce) {
        if (combine_block(kind, terms, RCELL(W, x, j0), RCELL(W, x, j0), RCELL(M, x, j0), len)) rc = -1;
      } else {
        memcpy(RCELL(W, x, j0), RCELL(M, x, j0), (size_t)len * ES);
      }
    }
    if (trace && step < ORC_MAX_STEPS) {
      trace->step_peer[step] = -1;
      trace->pulls[step] = 1;
      trace->combines[step] = reduce ? 1 : 0;
    }
  }
  for (int32_t x = 0; x < P; ++x)
    for (int64_t j = 0; j < ncols; ++j)
      memcpy((char*)out + ((int64_t)x * out_rank_stride + j) * ES, RCELL(W, x, j), ES);
#undef RCELL
  free(W); free(M);
  return rc;
}

/*
 * Independent instances (one Allreduce per instance, each with its own
 * block partition of n).  Layout of in and out: rank-major [P][batch][n].
 */
int oracle_allreduce_batched_ex(int32_t P, int64_t n, int32_t k, int32_t kind, int32_t group, int32_t schedule,
                                const void* in, void* out, int64_t batch) {
  if (kind == ORC_TERM || batch < 0) return -1;
  for (int64_t t = 0; t < batch; ++t) {
    int rc = oracle_allreduce_ex(P, n, k, kind, group, schedule, (const char*)in + t * n * 4, batch * n,
                                 (char*)out + t * n * 4, batch * n, NULL, n, NULL, NULL);
    if (rc) return rc;
  }
  return 0;
}

int oracle_allreduce_batched(int32_t P, int64_t n, int32_t k, int32_t kind,
                             const void* in, void* out, int64_t batch) {
  return oracle_allreduce_batched_ex(P, n, k, kind, ORC_GROUP_CYCLIC, ORC_SCHED_BUTTERFLY, in, out, batch);
}

/* ------------------------------------------------------------------------ */
/* The plain definition                                                      */
/* ------------------------------------------------------------------------ */

/* out[j] = sum over y of in[y][j], in fp64, ranks in increasing order. */
int oracle_direct_sum_f64(int32_t P, int64_t ncols, const float* in, int64_t in_rank_stride, double* out) {
  if (P < 1) return -1;
  for (int64_t j = 0; j < ncols; ++j) {
    double acc = 0.0;
    for (int32_t y = 0; y < P; ++y) acc += (double)in[(int64_t)y * in_rank_stride + j];
    out[j] = acc;
  }
  return 0;
}

/* out[j] = sum over y (wrapping modulo 2^32) or max over y of in[y][j]. */
int oracle_direct_i32(int32_t P, int64_t ncols, int32_t kind, const int32_t* in, int64_t in_rank_stride,
                      int32_t* out) {
  if (P < 1 || (kind != ORC_I32_SUM && kind != ORC_I32_MAX)) return -1;
  for (int64_t j = 0; j < ncols; ++j) {
    uint32_t s = 0;
    int32_t m = in[j];
    for (int32_t y = 0; y < P; ++y) {
      int32_t v = in[(int64_t)y * in_rank_stride + j];
      s += (uint32_t)v;
      if (v > m) m = v;
    }
    out[j] = kind == ORC_I32_SUM ? (int32_t)s : m;
  }
  return 0;
}

/* out[j] = max over y of in[y][j] (fp32; exact, order-independent). */
int oracle_direct_max_f32(int32_t P, int64_t ncols, const float* in, int64_t in_rank_stride, float* out) {
  if (P < 1) return -1;
  for (int64_t j = 0; j < ncols; ++j) {
    float m = in[j];
    for (int32_t y = 1; y < P; ++y) {
      float v = in[(int64_t)y * in_rank_stride + j];
      if (v > m) m = v;
    }
    out[j] = m;
  }
  return 0;
}

int32_t oracle_trace_size(void) { return (int32_t)sizeof(oracle_trace); }
