/*
 * rip.h -- C ABI of librip, a single-GPU (MI355X, gfx950) implementation of
 * Partial All-Reduce (P-Reduce) with a fused local update, the data-parallel
 * hot path of "Heterogeneity-Aware Asynchronous Decentralized Training"
 * (Ripples; arXiv 1909.08029).
 *
 * N model replicas ("workers") live in one GPU's memory.  One training step
 * of the algorithm of Fig. 4 is, for every worker i that computes this step:
 *   Step 2  x_i <- x_i - lr * grad_i            (optionally with momentum)
 *   Step 3  obtain a group G containing i        (rip_schedule_groups)
 *   Step 4  xbar = (1/|G|) sum_{g in G} x_g;  x_g <- xbar for all g in G
 *                                                (rip_preduce)
 * Groups that share no worker commute and run together in one launch
 * (Sec. 3.2, last paragraph).
 *
 * Conventions for every call below
 *  - Return value: RIP_OK (0) or a negative RIP_E_* code.  On error nothing
 *    is launched and no caller memory is written, except that the message
 *    returned by rip_last_error() is replaced (and except a HIP failure of
 *    the second launch of a split step; see rip_preduce).  No C++ exception
 *    crosses the boundary.
 *  - Host arrays passed in are read during the call only; the caller may
 *    reuse them as soon as the call returns.
 *  - Device buffers (parameters, gradients, momentum) belong to the caller.
 *    The library never allocates, frees or keeps them beyond the work it
 *    enqueues; the caller keeps them alive until the stream passes that work.
 *  - `stream` is a hipStream_t (NULL = the legacy default stream).  Device
 *    work is asynchronous on that stream.
 *  - Handles are not thread-safe; use one handle per thread or lock.
 *  - Graph capture: rip_local_step and rip_preduce enqueue one kernel
 *    launch (two for a step that mixes unit shapes with far-apart residency
 *    preferences; nothing when the step has no work), each with its part of
 *    the step -- schedule, optimizer scalars, the handle's pointer table --
 *    in the kernel argument, and no memset, copy or allocation.  They may be
 *    called on a stream under HIP graph capture; each replay re-applies the
 *    captured step to whatever the buffers hold then.  The replicas handle
 *    must outlive the graph.
 */
#ifndef RIP_H
#define RIP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RIP_ABI_VERSION 2

/* status codes */
enum {
  RIP_OK = 0,
  RIP_E_INVAL = -1,        /* bad argument: null pointer, size, id out of range,
                              group not strictly ascending, duplicate active id,
                              steps not consecutive, exhausted script */
  RIP_E_ALIGN = -2,        /* a device buffer is not 16-byte aligned */
  RIP_E_OVERLAP = -3,      /* one replica appears in two groups of one call,
                              or a registered buffer that a step writes
                              overlaps another registered buffer */
  RIP_E_UNSUPPORTED = -4,  /* unknown dtype or mode, or a size above a limit */
  RIP_E_HIP = -5,          /* HIP runtime error (text in rip_last_error) */
  RIP_E_NOMEM = -6         /* host or device allocation failed */
};

/* storage types of parameters, gradients and momentum; arithmetic is fp32 */
enum { RIP_FP32 = 0, RIP_BF16 = 1 };

/* Largest number of replicas one handle or scheduler accepts. */
#define RIP_MAX_REPLICAS 256

/* Message describing the last error on the calling thread ("" if none). */
const char* rip_last_error(void);
int32_t rip_abi_version(void);
/* Kernel launches the calling thread's last rip_preduce, rip_local_step or
 * rip_step enqueued: 0 (an error before any launch, or a step with no work),
 * 1, or 2 (a step split by residency preference; see rip_preduce).  For
 * accounting and tests; results never depend on it. */
int32_t rip_last_launch_count(void);

/* ------------------------------------------------------------------------
 * Group generation (Step 3 of Fig. 4; Sec. 4 and Sec. 5.1-5.3)
 *
 * The scheduler is a stepped model of the paper's Group Generator.  Each
 * worker keeps a request counter c_i (Sec. 5.3) and a Group Buffer, the
 * ordered list of groups that include it (Sec. 5.1).  One call per step t:
 *  1. Active workers = eligible this step and not blocked in a P-Reduce;
 *     they run their local update this step.
 *  2. Each active worker, in ascending id order (the Group Generator serves
 *     requests one at a time), asks for a group:
 *       TABLE / STATIC / RULE: the group of row (c_i - 1) mod period that
 *         contains it (a static schedule, Sec. 4.2, Fig. 8, Fig. 9); a worker
 *         with no group in that row skips synchronization (Sec. 4.2);
 *       RANDOM_GB / GD / INTER_INTRA / SCRIPTED: the head of its Group
 *         Buffer if that is not empty; else new groups are made and appended
 *         to the buffer of every member: one random group containing it
 *         (RANDOM_GB, Step 3 of Fig. 4), a random partition of all idle
 *         workers (Global Division, Sec. 5.1) admitting only workers w with
 *         c_i - c_w < c_thres when c_thres > 0 (Sec. 5.3), the two-phase
 *         Inter-Intra division (Sec. 5.2), or the next group of a script.
 *  3. A group runs when it heads every member's buffer and every member is
 *     blocked in it (serialization of conflicting groups, Sec. 4.1).  The
 *     groups that run are therefore disjoint.  Their members unblock.
 *
 * Random draws: SplitMix64 (Steele, Lea & Flood 2014) with keys folded as
 * k <- mix(k + 0x9E3779B97F4A7C15*(c+1)); bounded(n) = ((x>>32)*n)>>32.
 *   RANDOM_GB/GD/INTER_INTRA: one sequential stream from fold(seed, 3).
 *     RANDOM_GB group: k = min(kmin + bounded(kmax-kmin+1), N); the other
 *     k-1 members by a partial Fisher-Yates over the ascending ids != i
 *     (slot j swaps with j + bounded(N-1-j)).
 *     GD: Fisher-Yates over the ascending idle list (slot a swaps with
 *     bounded(a+1), a from the end), then consecutive chunks whose sizes are
 *     drawn as kmin + bounded(kmax-kmin+1) (the last chunk takes the rest).
 *   STATIC: row r of attempt a from its own stream fold(seed, 3, a, r): a
 *     Fisher-Yates shuffle of 0..N-1 cut into groups of group_size.  Attempts
 *     a = 0, 1, ... until the union of one period's groups connects all
 *     workers (the spectral-gap condition of Sec. 3.3); at most 1000.
 *   RULE: the rule table of Fig. 9: n_nodes nodes of 4 local workers, rank
 *     node*4 + local, period 4 (n_nodes = 1 or even).
 *   INTER_INTRA (Sec. 5.2): N/n_nodes consecutive workers per node.  A
 *     worker with an empty buffer divides the idle workers (same filter as
 *     GD): per node in ascending order a head = idle[bounded(count)]; the
 *     heads (ascending node order), then each node's other idle workers, are
 *     Fisher-Yates shuffled and cut into chunks as in GD (inter phase); then
 *     each node's idle workers form one group (intra phase).  Every idle
 *     worker thus gets its inter group, then its intra group, in its buffer.
 *   ADPSGD (the baseline of Fig. 3, for comparison on the same kernel): each
 *     active worker i draws x = bounded(N-1) and pairs with j = x (x < i) or
 *     x + 1; j is passive and need not be waiting.  Waiting requesters are
 *     then served oldest first; a pair runs unless one of its two workers
 *     is already in a pair of this step (the atomic averaging of Fig. 3),
 *     otherwise the requester keeps waiting.  Groups come out in request
 *     order; only requesters count requests and syncs.  N = 1: every
 *     request is a skip.
 * ---------------------------------------------------------------------- */
enum {
  RIP_SCHED_TABLE = 0,      /* caller's periodic table (FIXED = one row)   */
  RIP_SCHED_STATIC = 1,     /* seeded conflict-free periodic table         */
  RIP_SCHED_RANDOM_GB = 2,  /* random group per request + Group Buffers    */
  RIP_SCHED_GD = 3,         /* Global Division (+ slowdown filter)         */
  RIP_SCHED_SCRIPTED = 4,   /* Group Buffers fed by a caller's group list  */
  RIP_SCHED_RULE = 5,       /* the rule table of Fig. 9                    */
  RIP_SCHED_INTER_INTRA = 6,/* Inter-Intra division (Sec. 5.2)             */
  RIP_SCHED_ADPSGD = 7      /* AD-PSGD pairs with a passive partner (Fig. 3) */
};

typedef struct rip_sched rip_sched; /* opaque, library-owned */

typedef struct rip_sched_cfg {
  int32_t n_workers;   /* N, 1..RIP_MAX_REPLICAS */
  int32_t mode;        /* RIP_SCHED_* */
  uint64_t seed;       /* STATIC, RANDOM_GB, GD, INTER_INTRA, ADPSGD */
  int32_t group_size;  /* STATIC: N % group_size == 0, group_size >= 2 if N > 1 */
  int32_t period;      /* STATIC: rows per period (>= 1); TABLE: number of rows */
  int32_t kmin, kmax;  /* RANDOM_GB, GD, INTER_INTRA: 1 <= kmin <= kmax */
  int32_t c_thres;     /* GD, INTER_INTRA: slowdown threshold, <= 0 = off */
  int32_t n_nodes;     /* RULE: N == 4 * n_nodes; INTER_INTRA: N % n_nodes == 0 */
  /* TABLE: row r holds groups row_offsets[r] .. row_offsets[r+1]-1;
   * SCRIPTED: groups 0 .. n_groups-1 handed out in order.
   * Group g has members members[group_offsets[g] .. group_offsets[g+1]-1],
   * strictly ascending ids in [0, N); groups of one row are disjoint. */
  const int32_t* row_offsets;    /* TABLE: [period + 1], row_offsets[0] == 0 */
  const int32_t* group_offsets;  /* TABLE, SCRIPTED: [n_groups + 1] */
  const int32_t* members;        /* TABLE, SCRIPTED */
  int32_t n_groups;              /* TABLE, SCRIPTED */
} rip_sched_cfg;

/* Create a scheduler.  The configuration and its arrays are copied.
 * Errors: RIP_E_INVAL (sizes, table contents, a STATIC table with no
 * connected attempt), RIP_E_UNSUPPORTED (mode), RIP_E_NOMEM. */
int32_t rip_sched_create(const rip_sched_cfg* cfg, rip_sched** out);
void rip_sched_destroy(rip_sched* s); /* NULL is a no-op */

/* Schedule step `step`; steps must be 0, 1, 2, ... in order.
 *  eligible      [N] host bytes, nonzero = the worker finishes a local
 *                iteration this step if it is free; NULL = all eligible.
 *  active        out [N]: ascending ids of the workers updating this step
 *  n_active      out
 *  group_offsets out [N + 1], members out [N]: the groups that run this step
 *                as CSR, members ascending; ordered by creation (group-buffer
 *                modes) or by (iteration, position in the row) (table modes)
 *  n_groups      out
 * Output capacities are always enough: groups that run are disjoint.
 * Errors: RIP_E_INVAL (null handle or output, step out of order, a scripted
 * group that does not contain its requester, an exhausted script).  On an
 * error the scheduler state is unchanged. */
int32_t rip_schedule_groups(rip_sched* s, int64_t step, const uint8_t* eligible,
                            int32_t* active, int32_t* n_active,
                            int32_t* group_offsets, int32_t* members,
                            int32_t* n_groups);

typedef struct rip_worker_state {
  int64_t requests;  /* c_i: requests made (local iterations finished) */
  int64_t syncs;     /* groups of this worker that ran */
  int64_t skips;     /* requests with no group (table modes) */
  int32_t waiting;   /* 1 if blocked in a P-Reduce */
  int32_t gb_depth;  /* entries in its Group Buffer (ADPSGD: 1 while its pair waits) */
} rip_worker_state;

/* Counters of one worker; requests == syncs + skips + waiting always. */
int32_t rip_sched_worker(const rip_sched* s, int32_t worker, rip_worker_state* out);

/* ------------------------------------------------------------------------
 * Replicas: registered once, used by every step.
 *
 * Each replica r holds S segments (e.g. the layer tensors of a model; the
 * paper flattens them into one buffer per worker, Sec. 6.1 -- here they may
 * stay separate, or be views of one flat buffer).  Segment s has
 * seg_numel[s] elements in every replica.
 *  param  [N*S] host array of device pointers, param[r*S + s]
 *  grad   [N*S] or NULL (then only pure P-Reduce is possible)
 *  mom    [N*S] or NULL (momentum buffers, same storage type)
 * When every replica's non-empty segments lie back to back in memory (and
 * likewise for grad and mom), they are treated as one flat range and only
 * its first segment must be 16-byte aligned; otherwise every non-empty
 * segment must be.  Zero-length segments may be NULL.
 * Every non-empty segment must be device (or managed) memory of the current
 * device and lie inside the allocation holding its first byte; the buffers a
 * step writes (param, mom) must not overlap any other registered segment.
 * Gradient segments may overlap each other (replicas may share a gradient).
 * The handle copies the pointer table to device memory (one allocation,
 * freed by rip_replicas_destroy) on the current device; calls using it must
 * run with that device current.  Destroy only after the work that uses it
 * has finished.
 * Errors: RIP_E_INVAL (also: not device memory of this device, or a
 * segment running past its allocation), RIP_E_ALIGN, RIP_E_OVERLAP (a
 * written segment overlapping another), RIP_E_UNSUPPORTED (dtype, N above
 * RIP_MAX_REPLICAS), RIP_E_NOMEM, RIP_E_HIP. */
typedef struct rip_replicas rip_replicas; /* opaque, library-owned */

int32_t rip_replicas_create(int32_t n_replicas, int32_t n_segments, int32_t dtype,
                            const int64_t* seg_numel, void* const* param,
                            void* const* grad, void* const* mom, rip_replicas** out);
void rip_replicas_destroy(rip_replicas* r); /* NULL is a no-op */

/* For callers that cannot allocate device memory (code that runs while a HIP
 * graph is being captured, tight serving loops, harnesses that forbid
 * hipMalloc): the same registration as rip_replicas_create, with the same
 * arguments, checks and errors, but the handle's device tables (pointer
 * table and segment tables) go into a fixed array of RIP_NOALLOC_TABLE_BYTES
 * that the library keeps on each device for the life of the process, copied
 * there with a blocking hipMemcpy.  It calls no hipMalloc or hipFree.
 * Size: the tables take 24*N*S' + 8*S' + 32*(S'+1) bytes, where S' is 1 when
 * the segments are back to back (one flat range) and S otherwise; above the
 * array's size the call fails with RIP_E_UNSUPPORTED and changes nothing
 * (a failure of the copy itself, RIP_E_HIP, still supersedes the previous
 * handle).
 * Sharing: every such handle on a device uses that device's one array, which
 * keeps the last registration's tables.  Creating another one supersedes the
 * previous handle on that device: its later calls fail with RIP_E_INVAL
 * (destroying it is still fine).  A registration that overlaps work still in
 * flight with the previous handle on that device races with that work:
 * finish it (synchronize) first.  The handle is used and destroyed like any
 * other; handles from rip_replicas_create are unaffected.  The registration
 * itself copies synchronously, so it is made outside a stream capture; the
 * rip_preduce / rip_local_step / rip_step launches that use the handle may
 * then be captured like any others. */
#define RIP_NOALLOC_TABLE_BYTES 65536
int32_t rip_replicas_create_noalloc(int32_t n_replicas, int32_t n_segments, int32_t dtype,
                                    const int64_t* seg_numel, void* const* param,
                                    void* const* grad, void* const* mom, rip_replicas** out);

/* ------------------------------------------------------------------------
 * Local update and P-Reduce (Steps 2 and 4 of Fig. 4; F^G of Sec. 3.2)
 *
 * Arithmetic (fp32, this exact order; no fused multiply-add):
 *   active worker r:  g' = g_r + wd*w_r when weight_decay != 0, else g' = g_r;
 *                     u_r = w_r - lr*g', or with momentum
 *                     v_r = mu*v_r + g' (stored) and u_r = w_r - lr*v_r
 *                     (Nesterov: u_r = w_r - lr*(g' + mu*v_r))
 *   other worker r:   u_r = w_r
 *   group m1 < ... < mk:  s = u_m1; s = s + u_mj (j = 2..k, ascending);
 *                     xbar = s * (float)(1.0/k); w_m = xbar for every member
 *   active worker in no group: w_r = u_r
 *   every other replica: not read, not written.
 * bf16 storage: values widen exactly to fp32 and are rounded to nearest-even
 * once, when stored.  Momentum buffers are never averaged (Step 4 averages
 * parameters only).  momentum == 0 is plain SGD and leaves mom untouched.
 * The paper's ResNet-50 runs use momentum 0.9 and weight decay 1e-4
 * (Sec. 7.1.2); its VGG-16 runs plain SGD.
 * ---------------------------------------------------------------------- */
typedef struct rip_sgd {
  float lr;            /* learning rate (eta in Fig. 4) */
  float momentum;      /* mu; 0 = plain SGD.  Needs mom buffers when nonzero. */
  float weight_decay;  /* wd, added to the gradient as wd*w; 0 = none */
  int32_t nesterov;    /* nonzero: Nesterov momentum (needs momentum != 0) */
} rip_sgd;

/* Step 2 alone for the `n_active` workers listed in `active` (distinct ids).
 * Same as rip_preduce with no groups.
 * Errors: RIP_E_INVAL (null handle/sgd, ids, no grad or needed mom buffers,
 * Nesterov without momentum, device mismatch), RIP_E_UNSUPPORTED, RIP_E_HIP
 * as rip_preduce. */
int32_t rip_local_step(const rip_replicas* r, const int32_t* active, int32_t n_active,
                       const rip_sgd* sgd, void* stream);

/* Steps 2 and 4 fused in one pass over memory, for one step of the schedule:
 * the local update of every listed active worker, then the P-Reduce of each
 * of the `n_groups` groups given as CSR (group g = members[group_offsets[g]
 * .. group_offsets[g+1]-1], strictly ascending).  Groups must be disjoint
 * (RIP_E_OVERLAP otherwise).  sgd == NULL is pure P-Reduce; then n_active
 * must be 0.  One kernel launch covers all groups and updates, or, when the
 * step's units prefer residency caps far apart (a Global Division step of
 * pairs and groups of eight, say) and no cap is forced with
 * rip_set_blocks_per_cu, two launches in a row on `stream`, each at its own
 * cap; the units are disjoint, so the result is the same either way.  If the
 * second of two launches fails, the first has been enqueued (RIP_E_HIP).
 * Errors: RIP_E_INVAL (also: the current device is not the handle's),
 * RIP_E_OVERLAP, RIP_E_UNSUPPORTED (a step of 2^31 or more tiles), RIP_E_HIP
 * (launch failure). */
int32_t rip_preduce(const rip_replicas* r, const int32_t* group_offsets,
                    const int32_t* members, int32_t n_groups, const int32_t* active,
                    int32_t n_active, const rip_sgd* sgd, void* stream);

/* One whole step of the algorithm of Fig. 4 for every worker in one call:
 * group generation for `step` (Step 3, exactly as rip_schedule_groups with
 * the same arguments), then the fused local update and P-Reduce of the
 * groups that run (Steps 2 and 4, as rip_preduce with those groups and the
 * active workers).  Saves the host round trip between the two calls.
 *  s, r       scheduler and replicas handle with the same number of workers
 *  sgd        required (the workers that finish an iteration update); the
 *             handle needs gradient buffers, and momentum buffers when
 *             sgd->momentum != 0
 *  active .. n_groups  optional outputs, as in rip_schedule_groups (NULL =
 *             not wanted); written only on success
 * Atomic: on any error (including a failed launch) the scheduler is left as
 * it was, as if the call had not been made, and nothing is launched (a HIP
 * failure of the second launch of a split step leaves the first enqueued).
 * Errors: RIP_E_INVAL (null handle or sgd, worker counts differ, missing
 * buffers, Nesterov without momentum, device mismatch, a scheduling error),
 * RIP_E_HIP. */
int32_t rip_step(rip_sched* s, const rip_replicas* r, int64_t step, const uint8_t* eligible,
                 const rip_sgd* sgd, void* stream, int32_t* active, int32_t* n_active,
                 int32_t* group_offsets, int32_t* members, int32_t* n_groups);

/* Launch tuning (process-wide).  rip_set_max_blocks caps the workgroups of
 * one launch (0 = the default: one workgroup per tile up to 2^25
 * workgroups, beyond which workgroups loop over tiles); rip_set_blocks_per_cu
 * caps how many of the kernel's workgroups share a compute unit (0 = the
 * default: chosen per launch from its units' sizes, whether their members
 * update, and momentum, 4-14 per compute unit).  Negative values are
 * RIP_E_INVAL.  Results never depend on these settings. */
int32_t rip_set_max_blocks(int32_t max_blocks);
int32_t rip_set_blocks_per_cu(int32_t blocks_per_cu);

#ifdef __cplusplus
}
#endif

#endif /* RIP_H */
