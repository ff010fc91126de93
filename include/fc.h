/*
 * fc.h -- C ABI of the MI355X (gfx950) gradient-aggregation + SGD library.
 *
 * The operations follow the problem statement of FireCaffe (Iandola et al.,
 * arXiv 1511.00175):
 *   - Sec. 6 "Implementing efficient data parallel training": every worker
 *     computes the sum of weight gradients over its share of the batch, and
 *     the workers' sums are added together;
 *   - Sec. 6.2 "Reduction tree", Fig. 3b, Eq. 4: the element-wise sum is
 *     formed in binary reduction-tree order (branching factor 2, depth
 *     log2 p); Sec. 6.1 "Parameter server", Fig. 3a: the alternative adds all
 *     workers' vectors one after another at one node;
 *   - Fig. 3 caption and Sec. 6.1: the result is sent back to every worker,
 *     which applies the update to its local copy of the model;
 *   - Sec. 3 "Preliminaries", Sec. 7.1 item 2: batched SGD with momentum and
 *     weight decay.
 * On one GPU the K workers are K gradient replicas resident in device memory.
 *
 * Arithmetic (every operation one IEEE-754 binary32 op, round to nearest
 * even, no contraction, subnormals kept):
 *   s     = tree (or linear) sum over k of widen(grads[k][i])
 *   ga    = s * c,             c    = 1.0f / (float)batch (host, once)
 *   d     = ga + wd_j * w[i],  wd_j = wd * decay_mult_j
 *   v'    = mu * v[i] + lr_j * d,  lr_j = lr * lr_mult_j
 *   w'    = w[i] - v'
 * Tree shape for any K: neighbours are paired level by level and an odd last
 * node moves up unchanged (for K a power of two this is the balanced tree).
 *
 * Conventions for every entry point:
 *   - All buffers are device pointers owned by the caller; the library never
 *     frees or retains them beyond the call.  A plan owns only its own small
 *     device tables (tile map, segment multipliers, replica pointer tables).
 *   - Element i of a segment lives at element index i of every buffer (w, v,
 *     out, g, src, each replica, each broadcast destination); elements that
 *     belong to no segment are never written.
 *   - Every pointer must be 16-byte aligned (FC_EALIGN otherwise).
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream) and do not wait on the host (fc_plan_balance and
 *     fc_plan_read_timing do).  A call whose replica or destination pointers
 *     differ from the plan's previous call copies the new pointer table from
 *     host memory (the HIP runtime may finish that copy before returning).
 *     Calls on one plan must not run concurrently from several host threads.
 *   - Calls on one plan take effect in the order they are made, whatever
 *     their streams: a call on another stream than the plan's previous call
 *     first makes its stream wait, on the device, for the work enqueued so
 *     far on that previous stream (which must still exist), so the plan's
 *     tables and scratch never serve two calls at once.
 *   - Graph capture: a call whose replica and destination pointers equal
 *     the plan's previous call, with timing off, enqueues kernel launches
 *     only (no copies, no memsets, no waits), so it may be captured in a HIP
 *     graph; run it once eagerly first.  Whoever launches the graph orders
 *     its calls: a captured call neither waits for the plan's previous call
 *     nor becomes it.  A call that would replace a pointer table, or that has
 *     timing on, while its stream is capturing returns FC_EINVAL and
 *     enqueues nothing (use one plan per set of pointers in a graph).
 *   - Return value: FC_OK (0) or a negative error code (fc_strerror names
 *     it).  Argument errors are detected before anything is enqueued.
 */
#ifndef FC_H
#define FC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FC_OK 0
#define FC_EINVAL (-1) /* bad argument: null pointer, K out of range, bad table, batch < 1 */
#define FC_EALIGN (-2) /* pointer not 16-byte aligned, or a segment offset not a multiple of
                          4 elements */
#define FC_EALIAS (-3) /* a written buffer overlaps another buffer (see each call) */
#define FC_EHIP (-4)   /* the HIP runtime reported an error (allocation, copy or launch) */
#define FC_ENOMEM (-5) /* host allocation failed */
#define FC_ESIZE (-6)  /* fc_step_noalloc: the plan is larger than its fixed raw-sum array */

/* One segment = one layer's weight or bias block (Sec. 3, Eq. 1).  Offsets and
 * lengths are in elements.  Segments must be sorted by offset and must not
 * overlap; lengths may be zero or any size; the multipliers scale lr and wd
 * for this segment (1, 1 = uniform). */
typedef struct {
    uint64_t offset;
    uint64_t length;
    float lr_mult;
    float decay_mult;
} fc_segment;

/* Storage type of the gradient replicas.  Accumulation, weights, velocity,
 * the raw sum and broadcast copies are always fp32.  FC_F16 is the 16-bit
 * gradient storage named in Sec. 8.2 "Reducing communication among servers";
 * widening fp16 -> fp32 is exact. */
typedef enum { FC_F32 = 0, FC_F16 = 1 } fc_dtype;

/* Summation order: binary reduction tree (Sec. 6.2) or parameter-server
 * linear order (Sec. 6.1). */
typedef enum { FC_ORDER_TREE = 0, FC_ORDER_LINEAR = 1 } fc_order;

typedef struct fc_plan fc_plan;

/* How fc_step schedules the work (every schedule gives the same bits).
 * FUSED: one kernel reads the replicas and w, v and writes w', v'.
 * TWO_PASS: one kernel reduces into a raw-sum buffer, a second applies the
 *   update (on MI355X faster than FUSED when the replicas dominate the bytes,
 *   because HBM serves a replica stream with one write stream better than
 *   with two).
 * RESIDENT: one persistent launch, one block of 16 waves per compute unit;
 *   each block first reduces its share of the parameters on chip (HBM sees a
 *   pure read stream) and then updates them from there, so the raw sum never
 *   goes to HBM.  A block's share per round is what one compute unit holds:
 *   its LDS (1 KiB per 256-element tile: about 10 M parameters per round over
 *   256 compute units of 160 KiB), plus, when that saves rounds, the tiles
 *   its waves keep in registers (fp32 replicas in tiles of 2 vectors with
 *   K < 32: 0.8x as much again; fp16 replicas with K < 512: 0.4x); larger
 *   plans take several rounds, one launch per round.  It
 *   also makes fc_tree_reduce store the sums only after each read phase.
 *   Tiles of 64 lanes x 1 vector with batches of 16 replicas (default), or x 2
 *   vectors with batches of 4 (vecs_per_thread 2, K < 512).
 * RESIDENT_ONE_LAUNCH: RESIDENT with every round in one launch (the whole
 *   segment table in one kernel, whatever the plan's size): the persistent
 *   grid walks all its rounds itself, a block barrier
 *   between them, so fc_step and fc_tree_reduce are one launch each, and
 *   fc_broadcast one launch of grid x rounds blocks.  Same tiles, ranges and
 *   bits as RESIDENT (fc_plan_query reports this value); for a plan of one
 *   round the launches are the same.  With several rounds it is slower on
 *   MI355X (VGG-19 K=16 fp32, 8 rounds: 1802-1805 us per step vs 1763-1764
 *   us with one launch per round): within one launch the blocks drift apart,
 *   so one round's writes meet the next round's replica reads.
 * AUTO (no launch-shape field given): FUSED for a step of less than 64 MiB
 *   (n_elems * (K * bytes per element + 16)); otherwise RESIDENT when one
 *   round holds the plan or a parameter's replicas take at least 48 bytes
 *   (K * bytes per element), else FUSED.  With a launch-shape field: TWO_PASS when they take more than
 *   256 bytes, else FUSED. */
typedef enum {
    FC_SCHED_AUTO = 0,
    FC_SCHED_FUSED = 1,
    FC_SCHED_TWO_PASS = 2,
    FC_SCHED_RESIDENT = 3,
    FC_SCHED_RESIDENT_ONE_LAUNCH = 4
} fc_schedule;

/* Launch shape.  Results are bit-identical for every allowed setting; the
 * fields only change speed.  Zero selects the default, which depends on the
 * schedule, the replica type, K and the plan's size (measured on MI355X):
 * RESIDENT -> 64-lane tiles of (2 vectors, batches of 4 replicas) for fp32
 * replicas with K <= 16, else (1 vector, batches of 16); vecs_per_thread and
 * kchunk may name either; otherwise fp16 -> (4 vectors, 4 replicas, 256
 * threads); fp32 with K <= 4 -> (1, 8, 256); fp32 with 16 < K <= 64 ->
 * (4, 2, 256); other fp32 -> (1, 16, 64).  Replica loads always carry the
 * streaming (nt) hint. */
typedef struct {
    int block_threads;   /* 64, 128 or 256 threads per block */
    int vecs_per_thread; /* 4-element lane-vectors per thread (1, 2 or 4) ... */
    int kchunk;          /* ... and replicas loaded per batch; the pairs compiled are
                            (1, 8) (1, 16) (2, 8) (2, 16) (4, 2) (4, 4) (4, 8) */
    int max_blocks;      /* cap on the grid; blocks then loop over tiles (default: no cap) */
    int schedule;        /* fc_schedule of fc_step (default FC_SCHED_AUTO) */
    int k_waves;         /* 0 or 1: one wave reduces all K replicas of each of its
                            lane-vectors (other values are FC_EINVAL); 1 counts
                            as a launch-shape field for AUTO */
} fc_launch_opts;

/* Create a plan for K workers over a segment table (Sec. 6: one gradient
 * vector per worker).  segs[0..nseg-1] is copied; nseg may be 0 (every call
 * then does nothing).  1 <= K <= 1024.  Offsets must be multiples of 4
 * elements (16 bytes of fp32, 8 bytes of fp16).  Allocates the plan's device
 * tables on the current device with hipMalloc (FC_EHIP on failure); when
 * fc_step's schedule resolves to TWO_PASS the plan also owns a raw-sum
 * scratch buffer of 4 bytes per element of the segment extent.
 *   gdt   : an fc_dtype value, order: an fc_order value (plain ints, so that
 *           any value a caller passes is defined; others are FC_EINVAL)
 * On success *plan receives the plan; on failure *plan is set to NULL. */
int fc_plan_create(fc_plan** plan, const fc_segment* segs, int nseg, int K, int gdt, int order);

/* As fc_plan_create, with an explicit launch shape (NULL = defaults). */
int fc_plan_create_ex(fc_plan** plan, const fc_segment* segs, int nseg, int K, int gdt, int order,
                      const fc_launch_opts* opts);

/* Free the plan and its device tables (NULL is ignored).  The caller must
 * make sure no work that uses the plan is still running. */
void fc_plan_destroy(fc_plan* plan);

/* Reduce (Sec. 6.2, Fig. 3b; or Sec. 6.1 for FC_ORDER_LINEAR): for every
 * segment element i, out[i] = sum over k of widen(grads[k][i]), unscaled.
 *   grads : host array of K device pointers, replica k of the plan's dtype
 *   out   : device fp32 buffer.  It may be exactly grads[k] for an FC_F32
 *           plan (each element is read by the thread that writes it); any
 *           other overlap with a replica is FC_EALIAS. */
int fc_tree_reduce(fc_plan* plan, const void* const* grads, float* out, void* stream);

/* One momentum-SGD step with weight decay from a raw sum g (Sec. 3, Sec. 7.1
 * item 2; the averaging by 1/batch is the Sec. 6 equivalence with one GPU
 * summing over the whole batch):
 *   w, v : device fp32 weights and velocity, updated in place
 *   g    : device fp32 raw tree sum (as written by fc_tree_reduce)
 *   batch >= 1.  w, v and g must not overlap (FC_EALIAS). */
int fc_sgd_step(fc_plan* plan, float* w, float* v, const float* g, float lr, float mu, float wd,
                int batch, void* stream);

/* Send one fp32 vector back down the tree (Fig. 3 caption): dst[k][i] =
 * src[i] for every worker k < K and segment element i; other elements of the
 * destinations are not written.
 *   dst : host array of K device pointers.  No destination may overlap src
 *         or another destination (FC_EALIAS).
 * On a plan with the resident schedule it runs the plan's rounds of one
 * persistent block per compute unit (each block stages its range of src in
 * LDS and stores it one destination at a time); otherwise one block per
 * tile. */
int fc_broadcast(fc_plan* plan, const float* src, float* const* dst, void* stream);

/* The whole step in one pass over memory: reduce, average, SGD, write back,
 * and optionally keep the raw sum and broadcast w'.
 *   grads     : host array of K device replica pointers (plan's dtype)
 *   w, v      : device fp32 weights and velocity, updated in place
 *   out       : NULL, or a device fp32 buffer that receives the raw sum (it
 *               may be exactly grads[k] for an FC_F32 plan)
 *   bcast_dst : NULL, or a host array of K device fp32 pointers that
 *               receive w' (the workers' local model copies)
 * Result bits equal fc_tree_reduce, then fc_sgd_step, then fc_broadcast of w,
 * whatever the plan's schedule (in the two-pass schedule `out`, when given,
 * holds the raw sum between the passes; otherwise the plan's scratch does).
 * w, v, out and every destination must not overlap each other or a replica
 * (FC_EALIAS), except out == grads[k] as above. */
int fc_step(fc_plan* plan, const void* const* grads, float* w, float* v, float lr, float mu,
            float wd, int batch, float* out, float* const* bcast_dst, void* stream);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation: fc_step in
 * the two-pass schedule (a reduce pass into a raw-sum buffer, then the update
 * pass, which also stores the broadcast copies), whatever the plan's own
 * schedule, with the raw sum between the passes held in a fixed device array
 * of FC_NOALLOC_MAX_ELEMS floats (64 MiB) that the library reserves on each
 * GPU it runs on and keeps until the process ends.  Arguments, validation
 * and result bits are fc_step's.  When `out` is given it holds the raw sum
 * between the passes and the array is not used; otherwise the plan's extent
 * (one past its last segment element) must be at most FC_NOALLOC_MAX_ELEMS
 * (FC_ESIZE).  The current device must be the plan's (FC_EINVAL).  The call
 * allocates no device or host memory and records no per-kernel timing; like
 * every call it replaces a pointer table only when the pointers change.
 * Every call on one GPU uses that GPU's one array: calls that may run at the
 * same time on one GPU (other plans, other streams or threads) race on it;
 * calls on one plan are ordered (see the conventions above).  The array
 * needs no clearing: the reduce pass writes every segment element before the
 * update pass reads it. */
#define FC_NOALLOC_MAX_ELEMS 16777216
int fc_step_noalloc(fc_plan* plan, const void* const* grads, float* w, float* v, float lr, float mu,
                    float wd, int batch, float* out, float* const* bcast_dst, void* stream);

/* Learning-rate policies (Sec. 7.2 "Results: Midsized deep models", Sec. 7.3
 * "Results: Ultra-deep models").  The rate at iteration `iter` for a step of
 * `batch` samples is, evaluated in double and rounded to float once:
 *     lr = (base_lr * scale) * factor(iter)
 *     scale = batch / base_batch     (linear scaling with the batch, Sec. 7.2:
 *                                     4x the batch -> 4x the rate); 1 when
 *                                     base_batch == 0
 *     FIXED: factor = 1
 *     STEP : factor = gamma ^ floor(iter / stepsize)   (Sec. 7.2: divided by
 *            10 twice during training -> gamma 0.1)
 *     POLY : factor = (1 - iter / max_iter) ^ power    (Sec. 7.3, power 0.5),
 *            0 <= iter <= max_iter
 * pow() is the C library's. */
typedef enum { FC_LR_FIXED = 0, FC_LR_STEP = 1, FC_LR_POLY = 2 } fc_lr_kind;

typedef struct {
    int kind;          /* fc_lr_kind */
    int base_batch;    /* batch the base rate is quoted for; 0 = no batch scaling */
    double base_lr;    /* >= 0 */
    double gamma;      /* STEP: > 0 */
    int64_t stepsize;  /* STEP: >= 1 */
    int64_t max_iter;  /* POLY: >= 1 */
    double power;      /* POLY: >= 0 */
} fc_lr_policy;

/* *lr = the policy's rate at `iter` (>= 0) for `batch` (>= 1).  Host only;
 * FC_EINVAL for a bad policy or iteration. */
int fc_lr_at(const fc_lr_policy* policy, int64_t iter, int batch, float* lr);

/* Multi-step driver: n_iters fused steps (fc_step without raw sum or
 * broadcast) at iterations first_iter .. first_iter + n_iters - 1, each with
 * the policy's rate, all enqueued on `stream`.  The same K replicas feed every
 * step (a driver for benchmarks and tests; in training, call fc_lr_at and
 * fc_step once per iteration with that iteration's gradients).  Validation as
 * fc_step; stops at the first error. */
int fc_train(fc_plan* plan, const void* const* grads, float* w, float* v, const fc_lr_policy* policy,
             int64_t first_iter, int64_t n_iters, float mu, float wd, int batch, void* stream);

/* Read-bandwidth probe, for benchmarks: one streaming read of `bytes`
 * (a multiple of 16, > 0) from the device buffer `src` (16-byte aligned), the
 * access pattern that bounds any read-bound kernel on this GPU.  Every block
 * of 16 KiB stores one fp32 partial sum of its bytes read as fp32 into
 * out[block] (the rounding order is not specified; the sums only keep the
 * loads live), so `out` must hold fc_read_probe_blocks(bytes) floats.
 * Asynchronous on `stream`. */
uint64_t fc_read_probe_blocks(uint64_t bytes);
int fc_read_probe(const void* src, uint64_t bytes, float* out, void* stream);

/* Static description of a message code (never NULL). */
const char* fc_strerror(int code);

/* Plan facts for benchmarking and tests. */
typedef struct {
    int K;
    int nseg;
    int dtype;           /* fc_dtype */
    int order;           /* fc_order */
    uint64_t n_elems;    /* sum of segment lengths */
    uint64_t extent;     /* one past the last segment element */
    int ntiles;          /* blocks of work in one launch */
    int grid;            /* blocks launched (RESIDENT: its persistent grid) */
    int block_threads;   /* threads per block of the reduce or step launch */
    int vecs_per_thread;
    int kchunk;
    int schedule;        /* resolved fc_schedule of fc_step: FUSED, TWO_PASS, RESIDENT or
                            RESIDENT_ONE_LAUNCH (only when asked for) */
    uint64_t scratch_bytes; /* device memory the plan owns besides its tables */
    int k_waves;         /* always 1: one wave reduces all K replicas of a lane-vector */
    int lds_bytes;       /* RESIDENT: LDS per block (0 for the other schedules) */
    int rounds;          /* RESIDENT: rounds of the persistent grid (0 otherwise) */
} fc_plan_info;

int fc_plan_query(const fc_plan* plan, fc_plan_info* info);

/* Per-kernel timing, for benchmarks and tracing.  While enabled, every kernel
 * the plan launches is bracketed by two HIP events recorded on the launch
 * stream.  fc_plan_read_timing waits for the recorded events, returns per
 * kernel kind the number of launches and their summed duration (us) since
 * the previous read, and clears the record.  Enabling adds two event records
 * per launch and nothing else. */
enum { FC_KERNEL_STEP = 0, FC_KERNEL_REDUCE = 1, FC_KERNEL_SGD = 2, FC_KERNEL_BCAST = 3, FC_KERNEL_KINDS = 4 };

typedef struct {
    int launches[FC_KERNEL_KINDS];
    double total_us[FC_KERNEL_KINDS];
} fc_timing;

int fc_plan_set_timing(fc_plan* plan, int enable);
int fc_plan_read_timing(fc_plan* plan, fc_timing* timing);

/* XCD-aware shares for the RESIDENT schedule.  An MI355X runs the persistent
 * grid's blocks on 8 XCDs (block b on XCD b mod 8), and blocks on some XCDs
 * read HBM 6-10% more slowly than on others; every launch ends with its
 * slowest block.  Each resident launch adds, per block, the tiles it reduced
 * and the time its reduce phase took to a record the plan keeps, with the
 * XCD the block ran on (hardware register XCC_ID).  This call waits for
 * `stream` (a hipStream_t, NULL = the null stream: the stream of the plan's
 * calls), reads the record of every launch since the plan was made or last
 * balanced, clears it, and re-divides every round's tiles so that each
 * block's share is proportional to the tiles per second measured on its XCD,
 * drawn toward equal shares as far as needed for every share to fit a
 * block's LDS.  The stream of the plan's last call is drained too.  Only which block
 * reduces a tile changes: results are bit-identical before and after.  The
 * new shares apply to every later launch, including launches of graphs
 * captured before (the plan's device tables change in place; their sizes
 * and the launches' LDS do not).  It must not overlap any call of the same
 * plan on another stream.
 * xcd_rate (nullable): n_rate floats, entry x = XCD x's measured rate relative
 * to the mean over all blocks, 0 for an XCD that ran no block (at most 16 XCDs
 * are reported).  A plan that is not RESIDENT, whose blocks take fewer than
 * 32 tiles (of 256 elements) per round -- a launch of a few microseconds,
 * where the record would cost more than balancing gains, so nothing is
 * recorded -- or that has not launched since it was made or last balanced,
 * is left as it is (FC_OK, rates 0).  Errors: FC_EINVAL (NULL plan,
 * n_rate < 0, n_rate > 0 with xcd_rate NULL, or a stream it would wait on
 * being captured into a graph), FC_EHIP, FC_ENOMEM. */
int fc_plan_balance(fc_plan* plan, void* stream, float* xcd_rate, int n_rate);

#ifdef __cplusplus
}
#endif

#endif /* FC_H */
