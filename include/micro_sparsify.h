/*
 * micro_sparsify.h -- C ABI of the MI355X (gfx950) implementation of MiCRO's
 * per-worker gradient sparsification step (Yoon & Oh, arXiv 2310.00967).
 *
 * One call of micro_sparsify_step is one worker's share of one iteration of
 * the paper's Algorithm 1, restricted to the worker's own partition:
 *
 *   Sec. 4.1  partition:  [s, e) = [floor(r*N/n), floor((r+1)*N/n))
 *   Sec. 2    error feedback accumulation:  acc_j = grad_j + residual_j
 *             (one binary32 addition, round to nearest even, no fused
 *             multiply-add, subnormals kept)
 *   Sec. 4.2  exclusive selection:  j is selected iff |acc_j| >= theta
 *             (the binary32 magnitude compared with the binary64 threshold)
 *   Alg. 1    the selected pairs (j, acc_j), in increasing j, go to
 *             out_idx / out_val; residual_j becomes +0 where j is selected
 *             and acc_j elsewhere in [s, e)
 *   Sec. 4.3  threshold scaling:  theta <- Estimate(d * P, k, theta), in
 *             binary64 on the host from the selected count k
 *
 * Every function is extern "C", takes plain pointers and sizes, and reports
 * failure through micro_status; no C++ exception crosses the ABI.  Pointers
 * documented as "device" are HIP device addresses on the device that was
 * current when the context was created; "host" pointers are ordinary host
 * memory.  The caller owns every buffer it passes.
 *
 * Typical use, one worker of `world` over a gradient of n values already in
 * device memory (error handling shortened):
 *
 *   micro_ctx *ctx;
 *   micro_sparsify_init(&ctx, n, stream, NULL);          // NULL: default rule
 *   double theta = theta0;                               // e.g. a calibrated start
 *   for (int64_t t = 0; t < steps; ++t) {
 *       int32_t part; int64_t k;
 *       micro_cycle(t, worker, world, &part);            // Algorithm 1's rotation
 *       micro_sparsify_step(ctx, grad, residual, part, world, density, &theta,
 *                           out_idx, out_val, &k);       // out_* hold k pairs
 *       ... exchange out_idx[0, k) / out_val[0, k) with the other workers ...
 *   }
 *   micro_sparsify_free(ctx);
 */
#ifndef MICRO_SPARSIFY_H
#define MICRO_SPARSIFY_H

#include <stdint.h>

#if defined(__GNUC__)
#define MICRO_API __attribute__((visibility("default")))
#else
#define MICRO_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef struct micro_ctx micro_ctx; /* opaque, owned by the library */

typedef enum micro_status {
    MICRO_OK = 0,
    MICRO_EINVAL = 1,    /* an argument is invalid; nothing was modified        */
    MICRO_ECAPACITY = 2, /* a size exceeds what the context was created for     */
    MICRO_ERANGE = 3,    /* n_total does not fit int32 global indices           */
    MICRO_ENOMEM = 4,    /* a device or pinned host allocation failed           */
    MICRO_EHIP = 5       /* a HIP runtime call failed (see micro_last_error)    */
} micro_status;

/* Threshold update rules (readings of Sec. 4.3, which gives no formula). */
#define MICRO_RULE_PROPORTIONAL 0 /* theta * clamp(1 + beta*(k - k*)/k*, lo, hi) */
#define MICRO_RULE_FIXED_STEP 1   /* theta * (1 + alpha) if k > k*,
                                     theta * (1 - alpha) if k < k*, else theta   */
#define MICRO_RULE_HARD_THRESHOLD 2 /* theta never changes: the hard-threshold
                                       sparsifier the paper compares with
                                       (Sec. 1, Sec. 5.2), a fixed threshold  */
#define MICRO_RULE_TOPK 3 /* the exact top-k sparsifier the paper compares
                             with (Sec. 1: the k largest gradients; its density
                             footnote: d = k / n_g).  Not a threshold rule: the
                             step selects the k = max(1, floor(d * P)) values
                             of [s, e) whose accumulated magnitude is largest,
                             equal magnitudes by lower index, NaN never (so
                             fewer than k when fewer than k are not NaN).  The
                             incoming theta is not checked and does not change
                             the result: when it is positive and finite it is
                             a hint for the k-th magnitude (pass on the theta
                             the last step returned) and sets where the step
                             looks first.  theta receives the smallest
                             selected magnitude (0 or +inf possible; unchanged
                             when nothing is selected).  Through
                             micro_sparsify_step and micro_ef_step only
                             (MICRO_EINVAL in micro_sweep_step,
                             micro_sparsify_step_noalloc and
                             micro_estimate_threshold).  The k-th magnitude is
                             found by a radix select: three histogram passes
                             over the keys and a one-workgroup select after
                             each.  With a hint (and k <= P / 8, STAGED or
                             AUTO) the threshold step runs first at 7/8 of it
                             and the passes run over its output list, which
                             a trim then cuts to the top k; if that list holds
                             fewer than k values, they go back into the
                             residual and the select starts over on the
                             partition's residual.  Without one
                             the passes run over the partition first (waited
                             for), then the step at the k-th magnitude or at
                             the floor of its first digit, then the passes
                             left and the trim over its list.               */
#define MICRO_TOPK_ROUTE_FULL 1      /* micro_step_stats.topk_route: three passes over the partition, then the step */
#define MICRO_TOPK_ROUTE_LIST 2      /* one pass over the partition, the step, two passes over its list */
#define MICRO_TOPK_ROUTE_HINT_LIST 3 /* the step at the hint's bound, three passes over its list */
#define MICRO_TOPK_ROUTE_HINT_PICK 4 /* the step at the hint's bound listed fewer than k: one pass over the
                                        residual, then the values from the k-th magnitude's first-digit bin
                                        up extracted and two passes over them (or the passes and a pick
                                        over the residual) */

/* Kernel schedules (both compute the same result). */
#define MICRO_VARIANT_AUTO 0   /* per call, the faster measured schedule: TICKET
                                  for partitions of up to 2^20 values (one
                                  launch), STAGED above; both scratch sets     */
#define MICRO_VARIANT_TICKET 1 /* one pass; tiles from a ticket counter, each
                                  tile's offset by decoupled look-back           */
#define MICRO_VARIANT_STAGED 2 /* a streaming pass that stages each tile's pairs
                                  (no inter-workgroup waits), a scan pass (look-
                                  back per chunk of a million values) and a
                                  balanced pass that places them, the first two
                                  in one launch (see MICRO_FLAG_SEPARATE_SCAN);
                                  scratch of about 2 bytes per value of the
                                  vector                                          */

/* Flags. */
#define MICRO_FLAG_TIME_KERNEL 1 /* record HIP events around each launch so
                                    micro_sparsify_last_kernel_ms can report it */
#define MICRO_FLAG_SEPARATE_SCAN 2 /* STAGED: launch the scan pass on its own;
                                      by default micro_sparsify_step runs the
                                      streaming and scan passes as one launch
                                      (same result)                            */

typedef struct micro_config {
    int32_t rule;    /* MICRO_RULE_*                                  (default 0)    */
    double beta;     /* proportional gain                             (default 0.1)  */
    double lo, hi;   /* clamp of the proportional scale factor        (0.5, 2.0)     */
    double alpha;    /* fixed-step size                               (default 0.05) */
    int32_t variant; /* MICRO_VARIANT_*                               (default 0)    */
    int32_t flags;   /* MICRO_FLAG_*                                  (default 0)    */
} micro_config;

/* What the last micro_sparsify_step on a context did. */
typedef struct micro_step_stats {
    float kernel_ms;        /* device time of its kernels from HIP events
                               (MICRO_FLAG_TIME_KERNEL), else -1               */
    int64_t redone_tiles;   /* STAGED: 1024-value tiles with more selected
                               values than their staging slot holds (256),
                               redone by the placing pass instead              */
    int32_t variant;        /* the schedule the last step ran:
                               MICRO_VARIANT_TICKET or MICRO_VARIANT_STAGED    */
    int32_t fused;          /* 1 if its streaming and scan passes ran as one
                               launch (micro_sparsify_step, STAGED), else 0    */
    int32_t topk_route;     /* MICRO_RULE_TOPK: how the step found the k-th
                               magnitude (MICRO_TOPK_ROUTE_*); 0 for the other
                               rules, or when nothing was selectable           */
} micro_step_stats;

/* Fills *cfg with the defaults listed above. */
MICRO_API void micro_config_default(micro_config *cfg);

/*
 * Creates a context for flattened gradient vectors of n_total fp32 values on
 * the current HIP device, enqueuing all work on `hip_stream` (a hipStream_t;
 * NULL means the null stream).  cfg == NULL selects the defaults.
 * The context owns its device scratch (STAGED: a 256-pair staging slot and a
 * count per 1024 values of the vector plus look-back words, about 2 bytes per
 * value; TICKET: one look-back word per 4096 values; AUTO: both) and a pinned host word
 * for the selected count; it never owns the caller's buffers.
 * Returns MICRO_EINVAL (ctx NULL, n_total < 0, bad cfg), MICRO_ERANGE
 * (n_total > INT32_MAX: indices are int32), MICRO_EHIP (no usable device) or
 * MICRO_ENOMEM.  On failure *ctx is set to NULL.  Every context also holds
 * the top-k comparator's 8 KB of radix-select counters and 64 bytes of mapped
 * host memory.
 */
MICRO_API micro_status micro_sparsify_init(micro_ctx **ctx, int64_t n_total,
                                 void *hip_stream, const micro_config *cfg);

/*
 * One worker's sparsify step on partition `rank` of `world` (the paper's
 * cyclic partition number: the caller rotates it).
 *   grad      device, n_total fp32, read only; only [s, e) is read.
 *   residual  device, n_total fp32, in/out: the local error; only [s, e) is
 *             read and written, everything outside is untouched.
 *   rank, world  0 <= rank < world, world >= 1.
 *   density   the user-set density d, 0 < d <= 1; the target count is d*P.
 *   theta     host, in/out: the threshold of this step in, the threshold of
 *             the next step out.  Must be finite and > 0.  (MICRO_RULE_TOPK:
 *             the selection is the top k instead; theta in is unchecked and
 *             only a hint for where to look, theta out the k-th magnitude,
 *             see there.)
 *   out_idx   device int32, capacity >= P = e - s: the first k entries
 *             receive the selected global indices, strictly increasing.
 *   out_val   device fp32, capacity >= P: the first k entries receive acc
 *             at those indices.
 *   k         host out: the selected count.
 * The buffers grad[s,e), residual[s,e), out_idx[0,P) and out_val[0,P) must
 * not overlap.  grad and residual must be 4-byte aligned; the fastest path
 * needs them to share the same 16-byte phase.
 * The call is synchronous: it returns after the device work has finished and
 * theta has been updated.  Empty partitions (P == 0) return MICRO_OK with
 * k = 0 and theta unchanged.  Invalid arguments return MICRO_EINVAL before
 * any device work, with nothing modified.  A HIP failure returns MICRO_EHIP;
 * the outputs and the residual slice are then unspecified.
 * One context must not be used from two threads at once.
 */
MICRO_API micro_status micro_sparsify_step(micro_ctx *ctx, const float *grad,
                                 float *residual, int32_t rank, int32_t world,
                                 double density, double *theta,
                                 int32_t *out_idx, float *out_val, int64_t *k);

/*
 * micro_sparsify_step for callers that cannot allocate memory (tight serving
 * loops, harnesses that forbid hipMalloc, code that must not allocate after
 * start-up): no context, and no device or host allocation in the call.
 * It runs the one-pass schedule (MICRO_VARIANT_TICKET) with its scratch in
 * one static device array per device (4 MiB + 256 bytes, held from the first
 * call on a device until the process ends): a ticket counter, the count and
 * one look-back word per 4096 values of the partition, enough for any
 * partition of up to 2^31 - 1 values.
 *   grad, residual, rank, world, density, theta, out_idx, out_val, k:
 *              as micro_sparsify_step, over a vector of n_total values on
 *              the current HIP device; same results bit for bit.
 *   hip_stream a hipStream_t of the current device (NULL: the null stream);
 *              the call enqueues its kernel and the count readback there
 *              and waits for them.
 *   cfg        NULL for the defaults; only its threshold rule (rule, beta,
 *              lo, hi, alpha) is used.
 * Calls on one device share its scratch; the library serialises them (a lock
 * per device, held until the count is read back), so they never overlap on
 * it.  Returns MICRO_ERANGE for n_total above 2^31 - 1 (the most the scratch
 * covers), MICRO_EINVAL for the argument errors of micro_sparsify_step (and
 * an invalid cfg), MICRO_EHIP on a HIP failure; messages through
 * micro_last_error(NULL) on the calling thread.
 */
MICRO_API micro_status micro_sparsify_step_noalloc(const float *grad, float *residual, int64_t n_total,
                                                   int32_t rank, int32_t world, double density,
                                                   double *theta, int32_t *out_idx, float *out_val,
                                                   int64_t *k, void *hip_stream,
                                                   const micro_config *cfg);

/*
 * Every partition r of `world` (1 <= world <= 64) searched once over one
 * vector, each with its own threshold, in one set of launches (the streaming
 * and scan passes of all partitions as one launch for vectors of up to 64
 * scan chunks of a million values, unless MICRO_FLAG_SEPARATE_SCAN, then one
 * placing launch): the selections all n workers make at one iteration
 * (Sec. 4.2), with the local error of Sec. 2 / Eq. 1 reduced on the way.
 *   grad, residual  device, n_total fp32; residual in/out over all of it.
 *   theta      host double[world], in/out: theta[r] for partition r, then its
 *              next threshold (Sec. 4.3 over P_r).  Each finite and > 0.
 *   out_idx, out_val  device, n_total entries each: the selected (index, acc)
 *              pairs of all partitions, concatenated in index order, so
 *              partition r's pairs start at k[0] + ... + k[r-1].
 *   k          host int64[world], out: each partition's count.
 *   sumsq      host double[world] out, or NULL: the squared L2 norm of each
 *              partition's new residual, squares in binary64 added in a fixed
 *              order (within (P_r - 1) * 2^-53 relative of the exact sum);
 *              sqrt of their sum is the vector's local error norm.
 * The pairs, counts, thresholds and residual equal those of world calls of
 * micro_sparsify_step (rank 0 .. world-1) bit for bit.  Needs the staged
 * schedule.  Synchronous; errors as micro_sparsify_step (MICRO_EINVAL also
 * for world above 64 or the ticket variant).
 */
MICRO_API micro_status micro_sweep_step(micro_ctx *ctx, const float *grad, float *residual,
                                        int32_t world, double density, double *theta,
                                        int32_t *out_idx, float *out_val, int64_t *k,
                                        double *sumsq);

/* Algorithm 1 (cyclic assignment of partitions; Sec. 4.1): the partition
 * number that worker `worker` of `world` searches at iteration t,
 * ((t mod n) + worker) mod n (pure host arithmetic).  Returns MICRO_EINVAL
 * for NULL output, t < 0, world < 1 or worker outside [0, world). */
MICRO_API micro_status micro_cycle(int64_t t, int32_t worker, int32_t world, int32_t *cycle);

/*
 * Algorithm 1 for worker `worker` of `world` at iteration t over the whole
 * vector (the error-feedback accumulation of every element, then selection in
 * the worker's partition of this iteration only):
 *   c = micro_cycle(t, worker, world), [s, e) = partition c (Sec. 4.1);
 *   for every j in [0, n_total): acc = grad[j] + residual[j] (one binary32
 *   addition); j in [s, e) with |acc| >= theta is selected (its pair goes to
 *   the outputs, residual[j] = +0); every other j gets residual[j] = acc.
 *   theta <- Estimate(density * (e - s), k, theta) (Sec. 4.3).
 *   grad      device, n_total fp32, read only, all of it.
 *   residual  device, n_total fp32, in/out, all of it.
 *   out_idx, out_val, k, theta, density: as micro_sparsify_step, with
 *             P = e - s of partition c.
 *   cycle     host out (may be NULL): c.
 *   sumsq     host out (may be NULL): the squared L2 norm of the whole new
 *             residual, the worker's local error of Sec. 2 squared (Eq. 1
 *             averages its square root over the workers); squares in binary64
 *             added in a fixed order, within (n_total - 1) * 2^-53 relative of
 *             the exact sum (MICRO_RULE_TOPK with t values of the k-th
 *             magnitude left out of the selection: (n_total + t) * 2^-53).  Requesting it runs the pass through the sweep's
 *             kernels (the staged schedule; MICRO_EINVAL on a TICKET context).
 * grad[0, n), residual[0, n), out_idx[0, P) and out_val[0, P) must not
 * overlap.  Synchronous; errors as micro_sparsify_step.  A partition that is
 * empty (n_total < world) still accumulates every element, with k = 0 and
 * theta unchanged.
 */
MICRO_API micro_status micro_ef_step(micro_ctx *ctx, const float *grad, float *residual,
                                     int64_t t, int32_t worker, int32_t world, double density,
                                     double *theta, int32_t *out_idx, float *out_val,
                                     int64_t *k, int32_t *cycle, double *sumsq);

/*
 * Algorithm 1, after the all-gather of the selected indices: the worker's
 * accumulated values at the union of all workers' selections (its part of
 * the all-reduce) and their reset in its local error.
 *   residual   device, n_total fp32, in/out: the local error as
 *              micro_ef_step left it (acc at every unselected element).
 *   union_idx  device int32[m]: the union, distinct indices in [0, n_total);
 *              positions [own_first, own_first + own_count) hold this
 *              worker's own selection of the same iteration, in the order
 *              micro_ef_step wrote it (own_count = its k).
 *   own_val    device fp32[own_count]: micro_ef_step's out_val.
 *   out        device fp32[m], out: out[q] = acc at union_idx[q]
 *              (own_val[q - own_first] inside the own run).
 * Every union index outside the own run gets residual = +0 (those of the own
 * run already are).  An index outside [0, n_total) touches nothing and gives
 * out[q] = NaN.  Buffers must not overlap and must be 4-byte aligned.
 * Enqueued on the context's stream: the call returns after the launch (with
 * MICRO_FLAG_TIME_KERNEL it waits and records kernel_ms).  MICRO_EINVAL for
 * m outside [0, n_total], an own run outside [0, m), NULL or overlapping
 * buffers, before any device work.
 */
MICRO_API micro_status micro_union_gather(micro_ctx *ctx, float *residual, const int32_t *union_idx,
                                          int64_t m, int64_t own_first, int64_t own_count,
                                          const float *own_val, float *out);

/*
 * Algorithm 1 and Sec. 4.4, the model update with the averaged sums:
 * x[union_idx[q]] = x[union_idx[q]] - sums[q] / world for q in [0, m) (one
 * correctly rounded binary32 division by world, one binary32 subtraction;
 * the learning rate is inside the gradients).
 *   x          device, n_total fp32 model parameters, in/out.
 *   union_idx  device int32[m], distinct; indices outside [0, n_total) are
 *              skipped.
 *   sums       device fp32[m]: the all-reduced (summed) values.
 * Enqueued like micro_union_gather.  MICRO_EINVAL for m outside
 * [0, n_total], world < 1, NULL or overlapping buffers.
 */
MICRO_API micro_status micro_sparse_update(micro_ctx *ctx, float *x, const int32_t *union_idx,
                                           const float *sums, int64_t m, int32_t world);

/* Sec. 4.1 partition bounds (pure host arithmetic, no device needed):
 * *start = floor(rank*n_total/world), *len = floor((rank+1)*n_total/world)
 * - *start.  Returns MICRO_EINVAL for world < 1, rank outside [0, world),
 * n_total < 0 or NULL outputs. */
MICRO_API micro_status micro_partition(int64_t n_total, int32_t rank, int32_t world,
                             int64_t *start, int64_t *len);

/* Sec. 4.3 threshold update as the step applies it (pure host arithmetic):
 * *theta <- Estimate(density * part_len, k, *theta) under cfg (NULL =
 * defaults).  part_len == 0 leaves *theta unchanged.  Returns MICRO_EINVAL
 * for NULL theta, part_len < 0, k outside [0, part_len] or density outside
 * (0, 1]. */
MICRO_API micro_status micro_estimate_threshold(const micro_config *cfg, double density,
                                      int64_t part_len, int64_t k,
                                      double *theta);

/* The fp32 threshold the device compares with: the smallest binary32 value
 * >= theta (+inf when theta exceeds FLT_MAX).  For every binary32 x,
 * x >= *theta_f  <=>  (double)x >= theta, so the device's binary32 compare
 * selects exactly what the binary64 definition selects.  Returns
 * MICRO_EINVAL for NULL output or theta not finite and > 0. */
MICRO_API micro_status micro_threshold_f32(double theta, float *theta_f);

/* Copies the statistics of the last step on ctx (zeroes and kernel_ms = -1
 * before the first step or without MICRO_FLAG_TIME_KERNEL).  Returns
 * MICRO_EINVAL for NULL arguments. */
MICRO_API micro_status micro_sparsify_last_stats(const micro_ctx *ctx, micro_step_stats *stats);

/* Message of the last failure on ctx (or of the last failed init when ctx is
 * NULL); never NULL. */
MICRO_API const char *micro_last_error(const micro_ctx *ctx);

/* Static name of a status code. */
MICRO_API const char *micro_status_string(micro_status status);

/* Releases the context's scratch; NULL is a no-op.  Waits for the context's
 * stream first. */
MICRO_API void micro_sparsify_free(micro_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* MICRO_SPARSIFY_H */
