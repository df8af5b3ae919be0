/*
 * oracle_sanitize.c -- the CPU oracle run under AddressSanitizer and
 * UndefinedBehaviorSanitizer (gcc, host code only).
 *
 * Test infrastructure: links oracle/oracle.c and nothing of the HIP library.
 * Every rank row, output, column list and trace is its own heap allocation
 * of exactly the size the oracle is told, so a read or write past any of
 * them stops the run.  Over P = 1..64 and 72, 96, 127, 128, every k in
 * [L, 2L], the XOR group at power-of-two P and the Ring, with empty,
 * one-element, ragged and padded rows, it checks:
 *   - int32 sums (modulo 2^32) and maxima, fp32 maxima: equal to the plain
 *     definition, bit for bit, on every rank;
 *   - fp32 sums: within the worst-case bound of any summation order of P
 *     terms, gamma_{P-1} sum |x| with gamma_m = m u / (1 - m u), u = 2^-24
 *     (Higham, Accuracy and Stability of Numerical Algorithms, Sec. 4.2), of
 *     the fp64 sum;
 *   - a sample of columns gives the full run's values at those columns;
 *   - padding between strided rows is never written;
 *   - batched instances equal separate runs;
 *   - term mode: no combine of overlapping rank sets or of different blocks,
 *     every result covers all P ranks at its own block, and rendering into
 *     too small a buffer is refused without writing past it;
 *   - bad arguments return -1.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct orc_terms orc_terms;
orc_terms* oracle_terms_new(void);
void oracle_terms_free(orc_terms* t);
int64_t oracle_terms_violations(const orc_terms* t);
int64_t oracle_terms_count(const orc_terms* t);
void oracle_terms_mask(const orc_terms* t, int32_t id, uint64_t* out2);
int32_t oracle_terms_block(const orc_terms* t, int32_t id);
int64_t oracle_terms_render(const orc_terms* t, int32_t id, char* buf, int64_t cap);
int oracle_allreduce_ex(int32_t P, int64_t n, int32_t k, int32_t kind, int32_t group, int32_t schedule,
                        const void* in, int64_t in_rank_stride, void* out, int64_t out_rank_stride,
                        const int64_t* cols, int64_t ncols, orc_terms* terms, void* trace);
int oracle_allreduce_batched_ex(int32_t P, int64_t n, int32_t k, int32_t kind, int32_t group, int32_t schedule,
                                const void* in, void* out, int64_t batch);
int oracle_direct_sum_f64(int32_t P, int64_t ncols, const float* in, int64_t in_rank_stride, double* out);
int oracle_direct_i32(int32_t P, int64_t ncols, int32_t kind, const int32_t* in, int64_t in_rank_stride, int32_t* out);
int oracle_direct_max_f32(int32_t P, int64_t ncols, const float* in, int64_t in_rank_stride, float* out);
int32_t oracle_trace_size(void);

enum { I32_SUM = 0, I32_MAX = 1, F32_SUM = 2, F32_MAX = 3, TERM = 4 };
enum { CYCLIC = 0, XOR = 1 };
enum { BUTTERFLY = 0, RING = 1 };

static int fails = 0;
#define EXPECT(cond, ...)                               \
  do {                                                  \
    if (!(cond)) {                                      \
      if (fails < 40) {                                 \
        printf("FAIL (line %d): ", __LINE__);           \
        printf(__VA_ARGS__);                            \
        printf("\n");                                   \
      }                                                 \
      ++fails;                                          \
    }                                                   \
  } while (0)

static uint64_t rng_state = 88172645463325252ull;
static uint32_t next_u32(void) { /* xorshift64 (Marsaglia 2003) */
  rng_state ^= rng_state << 13;
  rng_state ^= rng_state >> 7;
  rng_state ^= rng_state << 17;
  return (uint32_t)(rng_state >> 16);
}

static int ceil_log2(int P) {
  int L = 0;
  while ((1 << L) < P) ++L;
  return L;
}

static void* xmalloc(size_t bytes) {
  void* p = malloc(bytes ? bytes : 1);
  if (!p) {
    printf("out of host memory\n");
    exit(2);
  }
  return p;
}

/* One replay with exactly sized rows ([P][stride] in one allocation, stride
 * >= n; padding filled with a sentinel that must survive in out). */
static void run_values(int P, int64_t n, int k, int group, int sched) {
  const int64_t stride = n + (P % 3);
  const size_t cells = (size_t)(P * stride);
  uint32_t* in = (uint32_t*)xmalloc(cells * 4);
  uint32_t* out = (uint32_t*)xmalloc(cells * 4);
  char what[96];
  snprintf(what, sizeof what, "P=%d n=%lld k=%d group=%d sched=%d", P, (long long)n, k, group, sched);
  for (int kind = 0; kind < 4; ++kind) {
    for (size_t i = 0; i < cells; ++i) {
      uint32_t v = next_u32();
      if (kind >= F32_SUM) { /* finite floats of mixed magnitude and sign */
        float f = ((float)(v >> 8) / 16777216.0f - 0.5f) * ldexpf(1.0f, (int)(v & 15) - 7);
        memcpy(&v, &f, 4);
      }
      in[i] = v;
      out[i] = 0xDEADBEEFu;
    }
    const int rc = oracle_allreduce_ex(P, n, k, kind, group, sched, in, stride, out, stride, NULL, n, NULL, NULL);
    EXPECT(rc == 0, "%s kind %d: rc %d", what, kind, rc);
    if (rc) continue;
    int bad = 0, pad = 0;
    for (int64_t j = 0; j < n; ++j) {
      if (kind == I32_SUM || kind == I32_MAX) {
        int32_t want;
        oracle_direct_i32(P, 1, kind, (const int32_t*)in + j, stride, &want);
        for (int x = 0; x < P; ++x) bad += (int32_t)out[x * stride + j] != want;
      } else if (kind == F32_MAX) {
        float want;
        oracle_direct_max_f32(P, 1, (const float*)in + j, stride, &want);
        for (int x = 0; x < P; ++x) bad += memcmp(&out[x * stride + j], &want, 4) != 0;
      } else {
        double exact, mag = 0.0;
        oracle_direct_sum_f64(P, 1, (const float*)in + j, stride, &exact);
        for (int y = 0; y < P; ++y) mag += fabs((double)((const float*)in)[y * stride + j]);
        const double nu = (P - 1) * ldexp(1.0, -24), bound = nu / (1.0 - nu) * mag * (1.0 + 1e-9);
        for (int x = 0; x < P; ++x) {
          float g;
          memcpy(&g, &out[x * stride + j], 4);
          bad += !(fabs((double)g - exact) <= bound);
        }
      }
    }
    for (int x = 0; x < P; ++x)
      for (int64_t j = n; j < stride; ++j) pad += out[x * stride + j] != 0xDEADBEEFu;
    EXPECT(bad == 0, "%s kind %d: %d results off the definition", what, kind, bad);
    EXPECT(pad == 0, "%s kind %d: %d padding cells written", what, kind, pad);

    /* a sample of columns: every third one, from an exactly sized list */
    if (n >= 3 && (kind == I32_SUM || kind == F32_SUM)) {
      const int64_t ns = (n + 2) / 3;
      int64_t* cols = (int64_t*)xmalloc((size_t)ns * 8);
      uint32_t* sin = (uint32_t*)xmalloc((size_t)(P * ns) * 4);
      uint32_t* sout = (uint32_t*)xmalloc((size_t)(P * ns) * 4);
      for (int64_t s = 0; s < ns; ++s) cols[s] = 3 * s;
      for (int x = 0; x < P; ++x)
        for (int64_t s = 0; s < ns; ++s) sin[x * ns + s] = in[x * stride + cols[s]];
      EXPECT(oracle_allreduce_ex(P, n, k, kind, group, sched, sin, ns, sout, ns, cols, ns, NULL, NULL) == 0,
             "%s: sampled run", what);
      int sb = 0;
      for (int x = 0; x < P; ++x)
        for (int64_t s = 0; s < ns; ++s) sb += sout[x * ns + s] != out[x * stride + cols[s]];
      EXPECT(sb == 0, "%s kind %d: %d sampled columns differ from the full run", what, kind, sb);
      free(cols);
      free(sin);
      free(sout);
    }
  }
  free(in);
  free(out);
}

/* Term mode: every result is a full tree over the P ranks at its block. */
static void run_terms(int P, int64_t n, int k, int group, int sched) {
  orc_terms* t = oracle_terms_new();
  int32_t* ids = (int32_t*)xmalloc((size_t)(P * n) * 4);
  void* trace = xmalloc((size_t)oracle_trace_size());
  const int rc = oracle_allreduce_ex(P, n, k, TERM, group, sched, NULL, n, ids, n, NULL, n, t, trace);
  EXPECT(rc == 0, "terms P=%d k=%d: rc %d", P, k, rc);
  if (rc == 0) {
    EXPECT(oracle_terms_violations(t) == 0, "terms P=%d k=%d group=%d sched=%d: %lld violations", P, k, group, sched,
           (long long)oracle_terms_violations(t));
    const int64_t q = n / P, m = n % P;
    int bad = 0;
    for (int x = 0; x < P; ++x)
      for (int64_t j = 0; j < n; ++j) {
        const int32_t id = ids[x * n + j];
        uint64_t mask[2];
        oracle_terms_mask(t, id, mask);
        const int cover = __builtin_popcountll(mask[0]) + __builtin_popcountll(mask[1]);
        /* column j lies in block b: the first m blocks hold q + 1 elements */
        const int64_t b = j < m * (q + 1) ? j / (q + 1) : m + (j - m * (q + 1)) / q;
        bad += cover != P || oracle_terms_block(t, id) != b;
      }
    EXPECT(bad == 0, "terms P=%d k=%d group=%d sched=%d: %d results miss ranks or blocks", P, k, group, sched, bad);
    /* rendering: the exact size fits, one byte less is refused */
    if (n > 0) {
      const int64_t cap0 = 64 * (int64_t)P * P + 64;
      char* big = (char*)xmalloc((size_t)cap0);
      const int64_t len = oracle_terms_render(t, ids[0], big, cap0);
      EXPECT(len > 0, "terms P=%d: render failed", P);
      if (len > 0) {
        char* fit = (char*)xmalloc((size_t)len + 1);
        char* tight = (char*)xmalloc((size_t)len);
        EXPECT(oracle_terms_render(t, ids[0], fit, len + 1) == len && strcmp(fit, big) == 0, "terms P=%d: exact fit", P);
        EXPECT(oracle_terms_render(t, ids[0], tight, len) == -1, "terms P=%d: a short buffer accepted", P);
        free(fit);
        free(tight);
      }
      free(big);
    }
  }
  free(trace);
  free(ids);
  oracle_terms_free(t);
}

static void bad_arguments(void) {
  int32_t in[64] = {0}, out[64];
  orc_terms* t = oracle_terms_new();
  EXPECT(oracle_allreduce_ex(0, 4, 0, I32_SUM, CYCLIC, BUTTERFLY, in, 4, out, 4, NULL, 4, NULL, NULL) == -1, "P = 0");
  EXPECT(oracle_allreduce_ex(129, 0, 8, I32_SUM, CYCLIC, BUTTERFLY, in, 0, out, 0, NULL, 0, NULL, NULL) == -1, "P = 129");
  EXPECT(oracle_allreduce_ex(5, 4, 2, I32_SUM, CYCLIC, BUTTERFLY, in, 4, out, 4, NULL, 4, NULL, NULL) == -1, "k < L");
  EXPECT(oracle_allreduce_ex(5, 4, 7, I32_SUM, CYCLIC, BUTTERFLY, in, 4, out, 4, NULL, 4, NULL, NULL) == -1, "k > 2L");
  EXPECT(oracle_allreduce_ex(6, 4, 3, I32_SUM, XOR, BUTTERFLY, in, 4, out, 4, NULL, 4, NULL, NULL) == -1, "XOR P = 6");
  EXPECT(oracle_allreduce_ex(4, 4, 6, I32_SUM, XOR, RING, in, 4, out, 4, NULL, 4, NULL, NULL) == -1, "Ring over XOR");
  EXPECT(oracle_allreduce_ex(4, 4, 5, I32_SUM, CYCLIC, RING, in, 4, out, 4, NULL, 4, NULL, NULL) == -1, "Ring k");
  EXPECT(oracle_allreduce_ex(4, 4, 3, 9, CYCLIC, BUTTERFLY, in, 4, out, 4, NULL, 4, NULL, NULL) == -1, "kind");
  EXPECT(oracle_allreduce_ex(4, -1, 3, I32_SUM, CYCLIC, BUTTERFLY, in, 4, out, 4, NULL, 0, NULL, NULL) == -1, "n < 0");
  EXPECT(oracle_allreduce_ex(4, 4, 3, I32_SUM, CYCLIC, BUTTERFLY, in, 4, out, 4, NULL, 3, NULL, NULL) == -1,
         "ncols != n without a column list");
  EXPECT(oracle_allreduce_ex(4, 4, 3, TERM, CYCLIC, BUTTERFLY, in, 4, out, 4, NULL, 4, NULL, NULL) == -1,
         "term mode without terms");
  EXPECT(oracle_allreduce_batched_ex(4, 4, 3, TERM, CYCLIC, BUTTERFLY, in, out, 1) == -1, "batched term mode");
  EXPECT(oracle_allreduce_batched_ex(4, 4, 3, I32_SUM, CYCLIC, BUTTERFLY, in, out, -1) == -1, "batch < 0");
  EXPECT(oracle_direct_i32(0, 1, I32_SUM, in, 1, out) == -1, "direct P = 0");
  EXPECT(oracle_direct_i32(2, 1, F32_SUM, in, 1, out) == -1, "direct i32 kind");
  EXPECT(oracle_terms_render(t, 0, (char*)out, 1) == -1, "render cap 1");
  oracle_terms_free(t);
  oracle_terms_free(NULL);
}

static void batched(int P, int64_t n, int k, int group, int sched, int64_t batch) {
  const size_t cells = (size_t)(P * batch * n);
  uint32_t* in = (uint32_t*)xmalloc(cells * 4);
  uint32_t* out = (uint32_t*)xmalloc(cells * 4);
  uint32_t* one_in = (uint32_t*)xmalloc((size_t)(P * n) * 4);
  uint32_t* one_out = (uint32_t*)xmalloc((size_t)(P * n) * 4);
  for (size_t i = 0; i < cells; ++i) in[i] = next_u32();
  EXPECT(oracle_allreduce_batched_ex(P, n, k, I32_SUM, group, sched, in, out, batch) == 0, "batched P=%d", P);
  int bad = 0;
  for (int64_t b = 0; b < batch; ++b) {
    for (int x = 0; x < P; ++x) memcpy(one_in + x * n, in + (x * batch + b) * n, (size_t)n * 4);
    oracle_allreduce_ex(P, n, k, I32_SUM, group, sched, one_in, n, one_out, n, NULL, n, NULL, NULL);
    for (int x = 0; x < P; ++x) bad += memcmp(one_out + x * n, out + (x * batch + b) * n, (size_t)n * 4) != 0;
  }
  EXPECT(bad == 0, "batched P=%d k=%d: %d instances differ from separate runs", P, k, bad);
  free(in);
  free(out);
  free(one_in);
  free(one_out);
}

static void sweep_p(int P, int term_pmax, int all_n) {
  const int L = ceil_log2(P);
  const int pow2 = (P & (P - 1)) == 0;
  const int64_t ns[4] = {2 * (int64_t)P + 3, 0, 1, P > 1 ? P - 1 : 2};
  const int nn = all_n ? 4 : 1;
  for (int k = L; k <= 2 * L; ++k) {
    for (int i = 0; i < nn; ++i) {
      run_values(P, ns[i], k, CYCLIC, BUTTERFLY);
      if (pow2) run_values(P, ns[i], k, XOR, BUTTERFLY);
    }
    if (P <= term_pmax) {
      run_terms(P, 2 * (int64_t)P + 1, k, CYCLIC, BUTTERFLY);
      if (pow2) run_terms(P, 2 * (int64_t)P + 1, k, XOR, BUTTERFLY);
    }
    if (P <= 16) batched(P, P + 2, k, CYCLIC, BUTTERFLY, 3);
  }
  for (int i = 0; i < nn; ++i) run_values(P, ns[i], 2 * (P - 1), CYCLIC, RING);
  if (P <= term_pmax) run_terms(P, 2 * (int64_t)P + 1, 2 * (P - 1), CYCLIC, RING);
  if (P <= 16) batched(P, P + 2, 2 * (P - 1), CYCLIC, RING, 3);
}

/* argv: the largest P of the full sweep (default 64), the largest P of the
 * term-mode checks (default 24); P = 72, 96, 127 and 128 follow with one
 * ragged n (the replay's cost grows like P^4 at the latency-optimal end). */
int main(int argc, char** argv) {
  const int pmax = argc > 1 ? atoi(argv[1]) : 64;
  const int term_pmax = argc > 2 ? atoi(argv[2]) : 24;
  bad_arguments();
  int swept = 0;
  for (int P = 1; P <= pmax && P <= 128; ++P, ++swept) sweep_p(P, term_pmax, 1);
  const int spots[4] = {72, 96, 127, 128};
  for (int i = 0; i < 4; ++i)
    if (spots[i] > pmax) {
      sweep_p(spots[i], term_pmax, 0);
      ++swept;
    }
  printf("%d values of P, %d failures\n", swept, fails);
  return fails != 0;
}
