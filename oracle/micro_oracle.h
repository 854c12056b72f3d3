/*
 * micro_oracle.h -- the CPU oracle for MiCRO's per-worker sparsify step.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, single-threaded C
 * implementation of what one worker computes in one iteration of MiCRO
 * (Yoon & Oh, "MiCRO: Near-Zero Cost Gradient Sparsification for Scaling and
 * Accelerating Distributed DNN Training", arXiv 2310.00967).  Only the tests,
 * the smoke check and the benchmark's CPU-baseline leg may load it.  It shares
 * no code, header or constant with the GPU library, and the GPU library never
 * calls it.
 *
 * What each function follows:
 *   micro_oracle_partition  Sec. 4.1 (coarse-grained partitioning): n equal
 *                           contiguous ranges of the flattened gradient.
 *   micro_oracle_select     Sec. 4.2 (exclusive gradient selection) and
 *                           Algorithm 1 (error-feedback accumulation, selection
 *                           in the worker's own partition, gathering the
 *                           accumulated values, zeroing the selected entries
 *                           and carrying the rest as the next local error),
 *                           with error feedback as described in Sec. 2.
 *   micro_oracle_estimate   Sec. 4.3 (compression ratio error minimisation by
 *                           threshold scaling) and the Estimate step of
 *                           Algorithm 1.  The paper gives no formula; the
 *                           reading implemented here is a memoryless
 *                           multiplicative scaling by the signed relative
 *                           compression ratio error, clamped.  Its form is
 *                           pinned by properties (direction, fixed point,
 *                           clamps, convergence of the density); the constants
 *                           beta, lo, hi and alpha are "parity unpinned"
 *                           against the paper, which prints none.
 *   micro_oracle_step       one worker, one iteration: the three above.
 *   micro_oracle_cycle      Algorithm 1 (cyclic assignment of partitions to
 *                           workers) and Sec. 4.1 (the assignment rotates at
 *                           the start of every iteration).
 *   micro_oracle_ef_step    Algorithm 1 for one worker over the whole
 *                           flattened vector: the error-feedback accumulation
 *                           of every element, selection only in the partition
 *                           of the worker's cycle, reset of the selected and
 *                           carry of every other element, then Estimate.
 *   micro_oracle_accumulate Algorithm 1, the accumulation of the new gradient
 *                           into the local error, for every element.
 *   micro_oracle_gather     Algorithm 1, the gathering of the accumulated
 *                           values at the globally selected indices.
 *   micro_oracle_zero       Algorithm 1, the reset of the accumulated values
 *                           at the globally selected indices.
 *   micro_oracle_update     Algorithm 1 and Sec. 4.4, the model update with the
 *                           averaged (all-reduced sum divided by n) values.
 *   micro_oracle_sumsq      Sec. 2 and Eq. 1: the square of the L2 norm of
 *                           (part of) the local error, the quantity the paper
 *                           averages over workers as its error measure.
 *   micro_oracle_sweep      every partition of one vector searched once, each
 *                           with its own threshold (the selections of all n
 *                           workers of Sec. 4.2 over one vector), with the
 *                           squared norm of each partition's local error.
 *
 * Precision: the accumulation is one binary32 addition (round to nearest even,
 * no fused multiply-add, subnormals kept); the threshold test compares the
 * magnitude, widened to binary64, against the binary64 threshold with ">=";
 * the threshold update is binary64 arithmetic.  Build with -ffp-contract=off
 * and without -ffast-math.
 */
#ifndef MICRO_ORACLE_H
#define MICRO_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Threshold update rules of the oracle (Sec. 4.3 readings). */
#define MICRO_ORACLE_PROPORTIONAL 0 /* theta * clamp(1 + beta*(k-k*)/k*, lo, hi) */
#define MICRO_ORACLE_FIXED_STEP 1   /* theta * (1 +/- alpha) by the sign of k-k* */

typedef struct micro_oracle_rule {
    int32_t kind;
    double beta;
    double lo;
    double hi;
    double alpha;
} micro_oracle_rule;

/* Fills the default rule: proportional, beta 0.1, clamp [0.5, 2], alpha 0.05. */
void micro_oracle_default_rule(micro_oracle_rule *rule);

/* Sec. 4.1.  Partition `rank` of `world` over [0, n_total): start = floor(rank*N/n),
 * end = floor((rank+1)*N/n).  Returns 0, or -1 for world < 1, rank outside
 * [0, world) or n_total < 0. */
int micro_oracle_partition(int64_t n_total, int32_t rank, int32_t world,
                           int64_t *start, int64_t *len);

/* Sec. 4.2 and Algorithm 1.  For j = start .. start+len-1 in increasing order:
 * acc = grad[j] + residual[j]; if |acc| >= theta, append (j, acc) to the
 * output lists and set residual[j] = +0; otherwise residual[j] = acc.
 * Returns the number k of appended pairs.  out_idx and out_val must hold len
 * entries.  Indices are global positions in the flattened vector. */
int64_t micro_oracle_select(const float *grad, float *residual, int64_t start,
                            int64_t len, double theta, int32_t *out_idx,
                            float *out_val);

/* Sec. 4.3.  Returns the next threshold from the target count
 * k* = density * part_len, the selected count k and the current threshold.
 * part_len == 0 returns theta unchanged. */
double micro_oracle_estimate(const micro_oracle_rule *rule, double density,
                             int64_t part_len, int64_t k, double theta);

/* One worker, one iteration: partition, select, estimate.  theta is in/out;
 * *k receives the selected count.  Returns 0, or -1 on invalid arguments
 * (in which case nothing is written). */
int micro_oracle_step(const float *grad, float *residual, int64_t n_total,
                      int32_t rank, int32_t world, double density,
                      const micro_oracle_rule *rule, double *theta,
                      int32_t *out_idx, float *out_val, int64_t *k);

/* Algorithm 1: the partition number that worker `worker` of `world` searches
 * at iteration t, ((t mod n) + i) mod n.  Over any n consecutive iterations a
 * worker visits every partition once, and at every iteration the workers'
 * partitions are all different (Sec. 4.1).  Returns -1 for t < 0, world < 1 or
 * worker outside [0, world). */
int32_t micro_oracle_cycle(int64_t t, int32_t worker, int32_t world);

/* Algorithm 1 for worker `worker` at iteration t, over the whole vector of
 * n_total values: for every j, acc = grad[j] + residual[j] (one binary32
 * addition); j inside the partition of the worker's cycle with |acc| >= theta
 * is selected (pair appended, residual[j] = +0), every other j keeps
 * residual[j] = acc.  Then theta = Estimate over the partition's length.
 * *cycle receives the partition number.  out_idx and out_val must hold the
 * partition's length.  Returns 0, or -1 on invalid arguments (nothing
 * written). */
int micro_oracle_ef_step(const float *grad, float *residual, int64_t n_total,
                         int64_t t, int32_t worker, int32_t world,
                         double density, const micro_oracle_rule *rule,
                         double *theta, int32_t *out_idx, float *out_val,
                         int64_t *k, int32_t *cycle);

/* Algorithm 1: acc[j] = grad[j] + residual[j] for j in [0, n) (binary32). */
void micro_oracle_accumulate(const float *grad, const float *residual,
                             int64_t n, float *acc);

/* Algorithm 1: out[q] = acc[idx[q]] for q in [0, m). */
void micro_oracle_gather(const float *acc, const int32_t *idx, int64_t m,
                         float *out);

/* Algorithm 1: acc[idx[q]] = +0 for q in [0, m). */
void micro_oracle_zero(float *acc, const int32_t *idx, int64_t m);

/* Algorithm 1 and Sec. 4.4: x[idx[q]] = x[idx[q]] - sums[q] / n for q in
 * [0, m): the all-reduced sum is averaged over the n workers (one binary32
 * division by n) and subtracted (one binary32 subtraction); the learning rate
 * is already inside the gradients.  The indices must be distinct.  Returns 0,
 * or -1 for world < 1. */
int micro_oracle_update(float *x, const int32_t *idx, const float *sums,
                        int64_t m, int32_t world);

/* Sec. 2 and Eq. 1: sum over j in [start, start+len) of residual[j]^2, each
 * square formed in binary64 (exact for a binary32 value) and added in index
 * order in binary64. */
double micro_oracle_sumsq(const float *residual, int64_t start, int64_t len);

/* Every partition r of `world` over one vector, in increasing r: the
 * partition step with threshold theta[r] (updated in place), its pairs
 * appended to out_idx/out_val after those of the partitions before it (so the
 * outputs are the concatenation in index order), k[r] its count, and, when
 * sumsq is not NULL, sumsq[r] = micro_oracle_sumsq over the partition after
 * its step.  out_idx and out_val must hold n_total entries.  Returns 0, or -1
 * on invalid arguments (nothing written). */
int micro_oracle_sweep(const float *grad, float *residual, int64_t n_total,
                       int32_t world, double density,
                       const micro_oracle_rule *rule, double *theta,
                       int32_t *out_idx, float *out_val, int64_t *k,
                       double *sumsq);

/* The exact top-k comparator (Sec. 1: sorting-based sparsifiers select the
 * k largest gradients; the density footnote: d = k / n_g) under the error
 * feedback of Sec. 2.  micro_oracle_topk_count returns the k of a range of len
 * values: floor(density * len) in binary64, at least 1, at most len; 0 when
 * len is 0. */
int64_t micro_oracle_topk_count(double density, int64_t len);

/* For j in [start, start+len): acc[j] = grad[j] + residual[j] (binary32).
 * The values ranked are the accumulated values that are not NaN, by |acc|
 * descending, equal magnitudes by increasing j; the first
 * min(k, number ranked) of them, k = micro_oracle_topk_count(density, len),
 * are selected.  Then, for j in increasing order: a selected j appends
 * (j, acc[j]) to the output lists and sets residual[j] = +0; every other j
 * sets residual[j] = acc[j].  *k_out receives the selected count and, when it
 * is positive, *kth the smallest selected magnitude (widened to binary64;
 * unchanged otherwise).  out_idx and out_val must hold len entries.  Returns
 * 0, or -1 on invalid arguments or a failed allocation (nothing written). */
int micro_oracle_topk_select(const float *grad, float *residual, int64_t start,
                             int64_t len, double density, int32_t *out_idx,
                             float *out_val, int64_t *k_out, double *kth);

#ifdef __cplusplus
}
#endif

#endif /* MICRO_ORACLE_H */
