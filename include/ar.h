/*
 * ar.h -- C ABI of the MI355X generalized Allreduce library (libar.so).
 *
 * The operation is Allreduce as defined in Kolmakov & Zhang, "A
 * Generalization of the Allreduce Operation" (arXiv:2004.09362), Sec. 1: P
 * ranks each own a vector of n elements; afterwards every rank holds the
 * elementwise combination of all P vectors.  Here the P ranks are virtual:
 * P device buffers on one GPU.  The schedule is the paper's permutation-group
 * algorithm over the cyclic group T_P with generator x -> x+1 (Sec. 5):
 *   - reduction phase of the bandwidth-optimal algorithm (Sec. 7), run once
 *     or, for fewer steps, shifted by s = 0 .. min(2^r, P)-1 (Sec. 8);
 *   - distribution phase: the reduction steps reversed without combination
 *     (Sec. 7), of which the first r are omitted (Sec. 8; r = ceil(log2 P)
 *     is the latency-optimal version of Sec. 9).
 * k_steps = 2*ceil(log2 P) - r, anywhere in [ceil(log2 P), 2*ceil(log2 P)].
 * ar_plan_create_ex adds the special cases the paper derives from the same
 * construction: the butterfly schedules over the group of Table 1b
 * (power-of-two P, t_k(x) = x XOR k), which are Recursive Halving (k = 2L,
 * Sec. 7), Recursive Doubling (k = L, Sec. 9) and their hybrid, and the Ring
 * (Sec. 6: cyclic group, operator t at every step, k = 2(P-1)).
 *
 * Conventions shared by all entry points:
 *   - Every function returns an ar_status; AR_OK is 0.  On failure nothing
 *     has been enqueued and ar_last_error_message() (per thread) describes
 *     it.
 *   - Device pointers are plain HIP device addresses on the current device.
 *     Host arrays (the table of rank pointers) are read during the call only.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL is the null stream)
 *     and the call returns without waiting.  Faults inside a kernel surface
 *     at the caller's next synchronisation.
 *   - The library never reads or writes host memory asynchronously and never
 *     falls back to a CPU path: without a usable GPU, execute calls return
 *     AR_ERR_NO_DEVICE.
 */
#ifndef AR_H_
#define AR_H_

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AR_OK = 0,
  AR_ERR_INVALID_ARG = 1,   /* bad P, n, k, pointer, batch or stride      */
  AR_ERR_UNSUPPORTED = 2,   /* dtype/op/path combination not provided     */
  AR_ERR_ALIAS = 3,         /* two rank buffers overlap                   */
  AR_ERR_OUT_OF_MEMORY = 4, /* workspace allocation failed                */
  AR_ERR_HIP = 5,           /* a HIP runtime call failed                  */
  AR_ERR_NO_DEVICE = 6,     /* no usable GPU                              */
  AR_ERR_INTERNAL = 7       /* the plan failed its own consistency check  */
} ar_status;

typedef enum { AR_INT32 = 0, AR_FLOAT32 = 1 } ar_dtype;

/* Combination function of Sec. 5.4.  AR_SUM on int32 wraps modulo 2^32.
 * AR_MAX keeps the received value only when it is strictly greater than the
 * kept one (so of -0.0 and +0.0 the kept value stays). */
typedef enum { AR_SUM = 0, AR_MAX = 1 } ar_op;

/* How ar_execute runs a plan.
 *   STEPWISE: one kernel launch per communication step of the schedule
 *             (2*ceil(log2 P) - r launches, plus one local copy when P = 2,
 *             k = 1), each pulling the peer's blocks out of HBM.  With
 *             blocks of at most 256 elements a launch streams each rank's
 *             run of consecutive blocks that share an operation as one
 *             flat space, so that batches of small instances fill waves.
 *   FUSED:    one launch that runs every step of the schedule on element
 *             columns held in registers, reading each input and writing
 *             each output once, for every plan with P >= 2: the Sec. 7 fold
 *             of a column (bandwidth-optimal), the primed and starred sums of
 *             Secs. 8-9 (fewer steps), the halving and doubling levels of the
 *             XOR group and the Ring's chain; latency-optimal cyclic plans
 *             with P <= 16 take a kernel without block tiling (many
 *             independent small instances, Sec. 1's 425-byte average).
 *             Sums whose blocks hold at most 64 elements (many small
 *             instances) run on flat columns, every rank's row loaded whole:
 *             cyclic plans with r < L and the Ring rotate each lane's column
 *             by its block before the same fold, recursion or chain; the
 *             XOR group's plans leave the block out (it only orders the
 *             operands of a halving pair, which a sum does not see).
 *             Otherwise, where every rank receives the same result
 *             (bandwidth-optimal plans, the Ring) and P >= 64, the launch
 *             stores each block's result on one rank and a second launch
 *             broadcasts it: one more block read and written per column,
 *             measured faster there.
 *   AUTO:     FUSED where it applies (P >= 2), STEPWISE otherwise.
 * Both paths combine exactly the same operand pairs in the same order, so
 * their results are bit-identical.
 *
 * Tuning overrides, read from the environment when a plan is created (they
 * change launch shapes and speed, never results):
 *   AR_STEP_NT, AR_FUSED_NT = 0|1   nontemporal loads and stores never /
 *                                   always (default: by bytes per launch);
 *   AR_STEP_MERGE = 0|1             step launches block by block / as
 *                                   merged runs of blocks (default: merged
 *                                   for blocks of at most 256 elements);
 *   AR_FUSED_SPLIT = 0|1            single fused launch, or reduce plus
 *                                   broadcast where every rank receives the
 *                                   same result (default: split for
 *                                   P >= 64, for P >= 24 when n * e is at
 *                                   least 32 MiB, and for P >= 33 in the
 *                                   rank-slot kernel);
 *   AR_BCAST_NT = 0|1               nontemporal loads and stores in that
 *                                   broadcast (default, for launches of 128
 *                                   MiB and more: the tiled copy with
 *                                   P >= 96 or on flat columns; the
 *                                   destination-major copy always);
 *   AR_BCAST_STREAM = 0|1|2|3       that broadcast tiled by block always /
 *                                   destination by destination wherever the
 *                                   call allows it (see fused_bcast_stream;
 *                                   default: the size rules given there),
 *                                   its chunks ordered by the default rule
 *                                   (1: one contiguous region of each slice
 *                                   per XCD on flat columns above 16 MiB per
 *                                   rank, on blocks that all start on the
 *                                   4 KB chunk grid for P >= 104 or from
 *                                   32 MiB per rank, and on other blocks
 *                                   for P >= 104 below 256 MiB per rank;
 *                                   else interleaved over the XCDs), always
 *                                   interleaved (2), or always in regions
 *                                   (3);
 *   AR_FUSED_PACKED = 0|1           column launches other than the latency-
 *                                   optimal ones: a wave takes 64 columns of
 *                                   one block of one instance, or one block
 *                                   of several instances when blocks hold at
 *                                   most 64 elements (default: the latter
 *                                   for batches with blocks that short);
 *   AR_FUSED_ROTATE = 0|1           sums (other than latency-optimal), and
 *                                   max in bandwidth-optimal, Ring and XOR
 *                                   plans:
 *                                   never / always on flat columns as above
 *                                   (default: when blocks hold at most 64
 *                                   elements; shifted sums at odd P >= 97
 *                                   or at P = 24-48 with n * e up to
 *                                   32 MiB; bandwidth-optimal and Ring
 *                                   plans from P = 33 with n * e below
 *                                   256 MiB; XOR-group plans other than
 *                                   Recursive Doubling at any length);
 *   AR_FUSED_CAP = N or N,M         resident workgroups per CU of the fused
 *                                   launch (and of the broadcast); 0 is no
 *                                   cap (default: per kernel and P);
 *   AR_LOG = 1                      print each plan (ar_plan_dump) to stderr
 *                                   when it is created. */
typedef enum { AR_PATH_AUTO = 0, AR_PATH_STEPWISE = 1, AR_PATH_FUSED = 2 } ar_path;

typedef struct ar_plan ar_plan; /* opaque; owned by the caller between create and destroy */

/* The group T_P of Sec. 5: AR_GROUP_CYCLIC, t_k(x) = (x + k) mod P (any P);
 * AR_GROUP_XOR, t_k(x) = x XOR k (Table 1b; P a power of two).  Placement p
 * of rank x holds block (x - p) mod P, respectively block x XOR p. */
typedef enum { AR_GROUP_CYCLIC = 0, AR_GROUP_XOR = 1 } ar_group;

/* AR_SCHEDULE_BUTTERFLY: the reduction / distribution schedules of Secs.
 * 7-9, k_steps in [L, 2L].  AR_SCHEDULE_RING: Sec. 6, cyclic group only,
 * k_steps = 2(P-1) (P - 1 reduction and P - 1 distribution steps, one block
 * per rank each). */
typedef enum { AR_SCHEDULE_BUTTERFLY = 0, AR_SCHEDULE_RING = 1 } ar_schedule;

/* Sizes of a plan (per Allreduce instance).  Block counts follow the paper's
 * cost equations (Secs. 7-9): a rank receives 2(P-1) blocks in the
 * bandwidth-optimal schedule, P*ceil(log2 P) in the latency-optimal one. */
typedef struct {
  int32_t P, L, k, r, w;             /* L = ceil(log2 P), r = 2L - k, w = min(2^r, P)   */
  int32_t rs_steps, ag_steps;        /* reduction / distribution steps; sum is k         */
  int32_t launches;                  /* kernel launches of the STEPWISE path              */
  int32_t fused_ok;                  /* 1 if the FUSED path can run this plan             */
  int64_t n, elem_bytes;
  int64_t blocks_pulled_per_rank;    /* same for every rank (translation invariance)     */
  int64_t bytes_pulled_per_rank_min; /* blocks differ by at most one element in length   */
  int64_t bytes_pulled_per_rank_max;
  int64_t bytes_pulled_total;        /* over all ranks = blocks_pulled_per_rank * n * e  */
  int64_t combines_per_rank;         /* block combinations                               */
  int64_t hbm_bytes_stepwise;        /* algorithmic HBM bytes of the STEPWISE path       */
  int64_t hbm_bytes_fused;           /* FUSED path: 2 * P * n * e (read every input, write
                                        every output), (2P + 1) * n * e when split       */
  int64_t workspace_bytes;           /* device scratch per instance, STEPWISE path       */
  int32_t group, schedule;           /* ar_group and ar_schedule of the plan              */
  int32_t fused_launches;            /* FUSED path: 1, or 2 when split into a reducing
                                        launch and a broadcast (every rank receives the
                                        same result and P >= 64; P >= 24 when n * e is
                                        at least 32 MiB; P >= 33 in the rank-slot
                                        kernel)                                          */
  int32_t fused_flat;                /* FUSED path with short blocks (sums; max in the
                                        bandwidth-optimal, Ring and XOR plans), and on
                                        long blocks the AR_FUSED_ROTATE defaults: 1
                                        when it runs on
                                        flat columns (the rank-slot kernel, or the XOR
                                        group's kernel without the block) for batches of
                                        fewer than 2^32 - 64 columns                     */
  int32_t exec_path;                 /* path ar_execute takes: AR_PATH_STEPWISE or
                                        AR_PATH_FUSED (AR_PATH_AUTO resolved); 0 when
                                        there is nothing to run (P = 1)                  */
  int64_t hbm_bytes_algorithmic;     /* algorithmic HBM bytes of the step-by-step
                                        schedule over all ranks (the paper's steps as
                                        separate passes: a combine reads two blocks and
                                        writes one, a copy reads and writes one); equal
                                        to hbm_bytes_stepwise                            */
  int32_t fused_bcast_stream;        /* FUSED path split into two launches: 1 when the
                                        broadcast of one instance copies destination by
                                        destination -- flat columns (short blocks), or
                                        blocks of at least 1024 elements in rank buffers
                                        of at least 2 MiB (AR_BCAST_STREAM overrides the
                                        size rule) -- for calls whose
                                        instances are contiguous (batch 1 or
                                        instance_stride = n) in 16-byte aligned rank
                                        buffers, with batch * n below 2^32 - 1024; other
                                        calls, and 0 here, take the tiled broadcast (the
                                        same bits)                                        */
} ar_stats;

/* One launch of the STEPWISE path: a list of placement ranges.  In a range,
 * every rank x works on placements p = p0 .. p0+count-1 (mod P); placement p
 * of rank x is block (x - p) mod P of its vector (Sec. 5.1 with h =
 * identity; x XOR p in the XOR group).  kind COPY: dst = src; REDUCE: dst =
 * own (+) src; REDUCE2: dst = own (+) src and dst2 = own2 (+) src.  own/dst
 * buffers belong to rank x, src to rank (x + delta) mod P (x XOR delta in the
 * XOR group); all at the same block.  Buffer ids: 0 is
 * the caller's rank buffer, 1 and 2 the plan's two scratch buffers, -1 none. */
typedef struct {
  int32_t phase;     /* 0 reduction, 1 distribution, 2 local copy */
  int32_t n_ranges;
} ar_launch_desc;

typedef struct {
  int32_t p0, count, kind, delta;
  int32_t dst, own, dst2, own2, src;
} ar_range_desc;

enum { AR_KIND_COPY = 0, AR_KIND_REDUCE = 1, AR_KIND_REDUCE2 = 2 };

/* k_steps value that asks plan creation to choose the step count (and the
 * path) from the cost model, as ar_plan_create_auto does with the default
 * parameters, one instance and the group of the call. */
#define AR_K_AUTO (-1)

/* Build the schedule for P ranks, n elements per rank and k_steps steps
 * (Secs. 7-9).  Host work only: validates, derives the per-step placement
 * ranges, assigns buffers, proves every launch free of read/write overlap
 * between ranks, and computes the sizes.  No device memory is touched.
 *   P in [1, 128]; n in [0, 2^46]; k_steps in [ceil(log2 P), 2*ceil(log2 P)]
 *   (k_steps = 0 for P = 1), or AR_K_AUTO; dtype/op from the enums above.
 * Errors: AR_ERR_INVALID_ARG (range), AR_ERR_UNSUPPORTED (dtype/op, or P
 * above the compiled maximum of 128), AR_ERR_INTERNAL (consistency check
 * failed).  *out_plan is set on AR_OK. */
ar_status ar_plan_create(int32_t P, int64_t n, ar_dtype dtype, ar_op op, int32_t k_steps, ar_plan** out_plan);

/* As ar_plan_create (which is group AR_GROUP_CYCLIC, schedule
 * AR_SCHEDULE_BUTTERFLY), for any group and schedule above.  Both paths
 * serve every plan; FUSED runs the whole schedule in one launch (Recursive
 * Halving / hybrid / Doubling: halving levels with the kept operand picked
 * per block, then doubling levels; Ring: the chain of Sec. 6), bit-identical
 * to STEPWISE.  Errors as ar_plan_create, and AR_ERR_INVALID_ARG for an
 * unknown group or schedule, AR_GROUP_XOR with P not a power of two, the
 * Ring over AR_GROUP_XOR, or a Ring k_steps other than 2(P-1).  AR_K_AUTO
 * is accepted for the butterfly schedules only. */
ar_status ar_plan_create_ex(int32_t P, int64_t n, ar_dtype dtype, ar_op op, int32_t k_steps, ar_group group,
                            ar_schedule schedule, ar_plan** out_plan);

/* Choose the execution path (default AR_PATH_AUTO).  AR_ERR_UNSUPPORTED if
 * FUSED is asked for and the plan cannot run fused. */
ar_status ar_plan_set_path(ar_plan* plan, ar_path path);

/* Allreduce in place (Sec. 1): afterwards every rank buffer holds the
 * elementwise combination (Sec. 5.4) of all P input vectors.  The schedule's
 * exchanges (Sec. 5.3: in a step, rank x receives the blocks of its peer
 * under the step's operator) are pulls here: the kernels of a step read the
 * peer's block out of HBM.  rank_buffers: host array of P device pointers, rank
 * x's n elements at rank_buffers[x].  Pointers must be 4-byte aligned and
 * must not overlap (AR_ERR_ALIAS); 16-byte aligned buffers take the
 * vectorised kernels.  With n = 0 nothing is touched and the pointers may be
 * NULL.  The first call on a plan that needs scratch (r > 0,
 * STEPWISE) allocates it on the current device; it is reused afterwards,
 * and a call that needs more (a larger batch or stride, another device)
 * allocates a larger one (at least twice the old on the same device, when
 * that much is free) and keeps the old one until ar_plan_destroy, so that
 * graphs captured before stay valid.  A plan must not run on two
 * streams at once (shared scratch).  An execute only enqueues kernels (no
 * memset, no synchronisation, no allocation once the scratch exists), so
 * after one call with the same device, batch and stride it may be captured
 * into a HIP graph; a captured call that would have to allocate returns
 * AR_ERR_UNSUPPORTED instead.  Graphs holding a plan's launches must not be
 * replayed after ar_plan_destroy. */
ar_status ar_execute(ar_plan* plan, void* const* rank_buffers, hipStream_t stream);

/* `batch` independent Allreduce instances per rank (Sec. 1's operation
 * applied to each; the exchanges of Sec. 5.3 as in ar_execute): instance j
 * of rank x is the n elements at rank_buffers[x] + j * instance_stride (in
 * elements, instance_stride >= n, (batch - 1) * instance_stride + n <= 2^46,
 * else AR_ERR_INVALID_ARG).  Each instance is split into blocks on its own.
 * Otherwise as ar_execute. */
ar_status ar_execute_batched(ar_plan* plan, void* const* rank_buffers, int64_t batch, int64_t instance_stride,
                             hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): ar_execute_batched
 * that never allocates.  Fused plans need no scratch; a step-wise plan with
 * r > 0 keeps its X and Y buffers in a device array inside the library
 * instead of the plan's scratch: 2 * P * round_up((batch - 1) *
 * instance_stride + n, 64) * 4 bytes must not exceed 64 MiB
 * (AR_ERR_UNSUPPORTED otherwise, nothing enqueued).  Each GPU that runs this
 * call holds that array from its first call until the process ends, and
 * every call on that GPU, from any plan or thread, shares it: calls that may
 * overlap on one GPU (other streams, other threads) race and must be
 * ordered by the caller.  Nothing in the array needs clearing: each call
 * writes every scratch element before reading it.  No hipMalloc, hipFree,
 * memset or host synchronisation; otherwise as ar_execute_batched.  The
 * first call on a device that needs the array looks up its address there
 * (hipGetSymbolAddress, which may load the library's device code): make that
 * call outside a graph capture. */
ar_status ar_execute_noalloc(ar_plan* plan, void* const* rank_buffers, int64_t batch, int64_t instance_stride,
                             hipStream_t stream);

/* Per-launch timing, for debugging and for measuring the per-step cost that
 * the model of Sec. 2 prices (alpha + beta*m + gamma*m per step).  As
 * ar_execute_batched, and in addition a timing-only HIP event (no
 * system-scope fence) is recorded on `stream` before the first launch and
 * after each launch.  The call then waits for the last event, so it returns
 * once the Allreduce has finished on the device.  The duration of launch i,
 * in milliseconds, is stored in launch_ms[i] for i < cap, and the number of
 * launches in *n_launches (0 when n = 0 or P = 1).  The events put a packet
 * between launches (a few microseconds each), so their sum exceeds the time
 * of an untimed execute by about that much.  Errors as ar_execute_batched;
 * AR_ERR_INVALID_ARG for a NULL n_launches, cap < 0, or a NULL launch_ms
 * with cap > 0; AR_ERR_HIP when an event call fails -- the launches are
 * then enqueued all the same (the Allreduce runs, in place), and
 * *n_launches is 0. */
ar_status ar_execute_timed(ar_plan* plan, void* const* rank_buffers, int64_t batch, int64_t instance_stride,
                           hipStream_t stream, float* launch_ms, int32_t cap, int32_t* n_launches);

/* Sizes of the plan; AR_ERR_INVALID_ARG for NULL arguments. */
ar_status ar_plan_stats(const ar_plan* plan, ar_stats* out);

/* Introspection of the STEPWISE launches (host side, for tests and tools):
 * number of launches, and launch i's description with up to `cap` ranges. */
ar_status ar_plan_num_launches(const ar_plan* plan, int32_t* out);

/* The plan as text: P, n, k, L, r, w, the step and block counts, the FUSED
 * path's kernel and choices, and the STEPWISE launch tables, one line per
 * launch.  Writes at most cap - 1 characters and a NUL into buf (nothing
 * when cap = 0), and the full length, without the NUL, into *len.  With
 * AR_LOG=1 in the environment, plan creation prints the same text to stderr.
 * AR_ERR_INVALID_ARG for a NULL plan or len, cap < 0, or a NULL buf with
 * cap > 0. */
ar_status ar_plan_dump(const ar_plan* plan, char* buf, int64_t cap, int64_t* len);
ar_status ar_plan_launch(const ar_plan* plan, int32_t i, ar_launch_desc* desc, ar_range_desc* ranges, int32_t cap);

/* Cost model (Sec. 2: a message of m bytes costs alpha + beta*m to send and
 * gamma*m to combine; u = m/P per block).  ar_model_time evaluates the
 * paper's cost equation for a k-step schedule of an m-byte vector over P
 * ranks: the bandwidth-optimal one (Sec. 7, k = 2L), the intermediate one
 * (Sec. 8, r = 2L - k removed steps) or the latency-optimal one (Sec. 9,
 * k = L), L = ceil(log2 P).  The Sec. 8 equation assumes the 2^r shifted
 * schedules do not wrap round the P placements; ar_plan_model_time prices
 * a plan's exact steps, blocks received and combinations instead, which
 * equal the equation's terms without wrap and fall below them with it.
 * ar_model_best_k returns the k in [L, 2L] with the smallest
 * ar_model_time, and the closed-form optimum r* of Sec. 8 (a real number;
 * NaN where its logarithms are undefined, e.g. P <= 2).
 * Errors: AR_ERR_INVALID_ARG for P outside [1, 128], k outside [L, 2L],
 * negative m/alpha/beta/gamma or NULL outputs. */
ar_status ar_model_time(int32_t P, double m_bytes, int32_t k_steps, double alpha, double beta, double gamma,
                        double* tau_seconds);
ar_status ar_model_best_k(int32_t P, double m_bytes, double alpha, double beta, double gamma, int32_t* k_steps,
                          double* r_closed_form);
ar_status ar_plan_model_time(const ar_plan* plan, double alpha, double beta, double gamma, double* tau_seconds);

/* The Sec. 2 model for this library's two ways of running a plan on one GPU,
 * where the P ranks share one HBM: a launch costs a fixed time (the paper's
 * alpha) plus its HBM bytes over a bandwidth.  STEPWISE runs one launch per
 * step and moves hbm_bytes_algorithmic (so with u bytes per block, a
 * received block costs about 2P*u / step_bytes_per_s and a combination
 * P*u / step_bytes_per_s: the paper's beta and gamma for P ranks on one
 * device); FUSED runs fused_launches launches moving hbm_bytes_fused.
 * Times are per call of ar_execute_batched with `batch` instances. */
typedef struct {
  double step_alpha;         /* seconds per step launch                          */
  double step_bytes_per_s;   /* HBM bytes per second of a step launch            */
  double fused_alpha;        /* seconds per fused launch                          */
  double fused_bytes_per_s;  /* HBM bytes per second of the fused launches        */
} ar_model_params;

/* Parameters fitted on MI355X (gfx950) by timing both paths over message
 * sizes (the library's calibration tool prints them for another device). */
ar_status ar_model_default_params(ar_model_params* out);

/* Model time of one call of ar_execute_batched on `plan` with `batch`
 * instances on `path` (AR_PATH_AUTO: the path ar_execute would take).
 * NULL params: the defaults.  AR_ERR_INVALID_ARG for NULL plan/output,
 * batch < 1, non-positive bandwidths or negative alphas; AR_ERR_UNSUPPORTED
 * for FUSED on a plan that cannot run fused. */
ar_status ar_plan_model_seconds(const ar_plan* plan, const ar_model_params* params, int64_t batch, ar_path path,
                                double* seconds);

/* Plan with the step count chosen by the cost model (Sec. 8 picks the
 * number of steps from alpha, beta and gamma measured on the machine;
 * Sec. 10 measures them): every k in [L, 2L] of the butterfly schedules is
 * priced on the STEPWISE path (ar_plan_model_seconds), and the cheapest k
 * is taken (the smallest on a tie).  With `path` AR_PATH_AUTO the plan then
 * runs FUSED if that path's model time is below the step-wise one at that
 * k, else STEPWISE; AR_PATH_STEPWISE or AR_PATH_FUSED fixes the path (every
 * fused plan moves the same bytes whatever k, so k still follows the
 * step-wise prices, the paper's choice).  The plan's results are those of
 * the chosen k (ar_plan_stats reports k and exec_path).  NULL params: the
 * defaults.  Errors as ar_plan_create_ex, AR_ERR_INVALID_ARG for batch < 1
 * or bad params, AR_ERR_UNSUPPORTED for FUSED with P = 1. */
ar_status ar_plan_create_auto(int32_t P, int64_t n, ar_dtype dtype, ar_op op, ar_group group, int64_t batch,
                              ar_path path, const ar_model_params* params, ar_plan** out_plan);

/* Wait for the plan's last stream, free its scratch and the plan.  NULL is
 * accepted.  Must not be called while another thread executes the plan. */
void ar_plan_destroy(ar_plan* plan);

/* Static text for a status code. */
const char* ar_status_string(ar_status s);

/* Detail of the last failure on the calling thread ("" if none), e.g. the
 * HIP error text.  The string stays valid until the thread's next call into
 * the library.  ar_last_error is the same function under a shorter name. */
const char* ar_last_error_message(void);
const char* ar_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* AR_H_ */
