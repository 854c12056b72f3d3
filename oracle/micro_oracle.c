/*
 * micro_oracle.c -- TEST INFRASTRUCTURE ONLY: the plain CPU oracle for
 * MiCRO's per-worker sparsify step (arXiv 2310.00967).  See micro_oracle.h
 * for what each function follows.  Deliberately a straight loop: no SIMD, no
 * threads, no blocking, no reordering.  Compile with -O2 -ffp-contract=off,
 * never with -ffast-math.
 */
#include "micro_oracle.h"

#include <math.h>
#include <stddef.h>
#include <stdlib.h>

void micro_oracle_default_rule(micro_oracle_rule *rule)
{
    rule->kind = MICRO_ORACLE_PROPORTIONAL;
    rule->beta = 0.1;
    rule->lo = 0.5;
    rule->hi = 2.0;
    rule->alpha = 0.05;
}

/* Sec. 4.1: the flattened gradient is divided into n equal contiguous ranges;
 * when n does not divide N, the floor split makes the lengths differ by at
 * most one and the ranges still tile [0, N) exactly. */
int micro_oracle_partition(int64_t n_total, int32_t rank, int32_t world,
                           int64_t *start, int64_t *len)
{
    if (world < 1 || rank < 0 || rank >= world || n_total < 0)
        return -1;
    int64_t s = ((int64_t)rank * n_total) / (int64_t)world;
    int64_t e = ((int64_t)rank * n_total + n_total) / (int64_t)world;
    *start = s;
    *len = e - s;
    return 0;
}

/* Sec. 4.2 and Algorithm 1: every element of the worker's own partition is
 * inspected.  The error-feedback accumulation adds the new gradient to the
 * local error (Sec. 2); an element whose accumulated magnitude reaches the
 * threshold is selected, its accumulated value is what the worker contributes,
 * and its local error restarts from zero; an unselected element keeps its
 * accumulated value as the next local error. */
int64_t micro_oracle_select(const float *grad, float *residual, int64_t start,
                            int64_t len, double theta, int32_t *out_idx,
                            float *out_val)
{
    int64_t k = 0;
    for (int64_t j = start; j < start + len; ++j) {
        float acc = grad[j] + residual[j];
        double mag = (double)fabsf(acc);
        if (mag >= theta) {
            out_idx[k] = (int32_t)j;
            out_val[k] = acc;
            k = k + 1;
            residual[j] = 0.0f;
        } else {
            residual[j] = acc;
        }
    }
    return k;
}

/* Sec. 4.3: the threshold of the next iteration is derived from the target
 * count k* and the count actually selected.  The paper states only that the
 * update inspects whether the selected count exceeds the target and assigns an
 * adjusted threshold; the proportional reading scales the threshold by one
 * plus beta times the signed relative compression ratio error, clamped to
 * [lo, hi]; the fixed-step reading moves it by a factor 1 +/- alpha. */
double micro_oracle_estimate(const micro_oracle_rule *rule, double density,
                             int64_t part_len, int64_t k, double theta)
{
    if (part_len == 0)
        return theta;
    double target = density * (double)part_len;
    double selected = (double)k;
    if (rule->kind == MICRO_ORACLE_FIXED_STEP) {
        if (selected > target)
            return theta * (1.0 + rule->alpha);
        if (selected < target)
            return theta * (1.0 - rule->alpha);
        return theta;
    }
    double rel_err = (selected - target) / target;
    double scale = rule->beta * rel_err;
    scale = 1.0 + scale;
    if (scale < rule->lo)
        scale = rule->lo;
    if (scale > rule->hi)
        scale = rule->hi;
    return theta * scale;
}

int micro_oracle_step(const float *grad, float *residual, int64_t n_total,
                      int32_t rank, int32_t world, double density,
                      const micro_oracle_rule *rule, double *theta,
                      int32_t *out_idx, float *out_val, int64_t *k)
{
    int64_t start = 0, len = 0;
    if (grad == NULL || residual == NULL || rule == NULL || theta == NULL ||
        k == NULL)
        return -1;
    if (micro_oracle_partition(n_total, rank, world, &start, &len) != 0)
        return -1;
    if (!(density > 0.0 && density <= 1.0))
        return -1;
    if (!(*theta > 0.0) || isinf(*theta))
        return -1;
    if (len > 0 && (out_idx == NULL || out_val == NULL))
        return -1;
    int64_t selected = micro_oracle_select(grad, residual, start, len, *theta,
                                           out_idx, out_val);
    *theta = micro_oracle_estimate(rule, density, len, selected, *theta);
    *k = selected;
    return 0;
}

/* Algorithm 1: the partition number advances by one for every worker at
 * every iteration, so the n workers always hold n different partitions and
 * each worker's search range covers the whole vector in n iterations. */
int32_t micro_oracle_cycle(int64_t t, int32_t worker, int32_t world)
{
    if (t < 0 || world < 1 || worker < 0 || worker >= world)
        return -1;
    int64_t n = (int64_t)world;
    return (int32_t)((t % n + (int64_t)worker) % n);
}

/* Algorithm 1 for one worker, element by element in index order: every
 * element accumulates its new gradient into the local error; only elements of
 * the worker's partition of this iteration are candidates for selection; a
 * selected element's accumulated value is contributed and its local error
 * restarts from zero, every other element carries its accumulated value. */
int micro_oracle_ef_step(const float *grad, float *residual, int64_t n_total,
                         int64_t t, int32_t worker, int32_t world,
                         double density, const micro_oracle_rule *rule,
                         double *theta, int32_t *out_idx, float *out_val,
                         int64_t *k, int32_t *cycle)
{
    int64_t start = 0, len = 0;
    if (grad == NULL || residual == NULL || rule == NULL || theta == NULL ||
        k == NULL || cycle == NULL)
        return -1;
    int32_t part = micro_oracle_cycle(t, worker, world);
    if (part < 0)
        return -1;
    if (micro_oracle_partition(n_total, part, world, &start, &len) != 0)
        return -1;
    if (!(density > 0.0 && density <= 1.0))
        return -1;
    if (!(*theta > 0.0) || isinf(*theta))
        return -1;
    if (len > 0 && (out_idx == NULL || out_val == NULL))
        return -1;
    int64_t selected = 0;
    for (int64_t j = 0; j < n_total; ++j) {
        float acc = grad[j] + residual[j];
        int inside = j >= start && j < start + len;
        if (inside && (double)fabsf(acc) >= *theta) {
            out_idx[selected] = (int32_t)j;
            out_val[selected] = acc;
            selected = selected + 1;
            residual[j] = 0.0f;
        } else {
            residual[j] = acc;
        }
    }
    *theta = micro_oracle_estimate(rule, density, len, selected, *theta);
    *k = selected;
    *cycle = part;
    return 0;
}

void micro_oracle_accumulate(const float *grad, const float *residual,
                             int64_t n, float *acc)
{
    for (int64_t j = 0; j < n; ++j)
        acc[j] = grad[j] + residual[j];
}

void micro_oracle_gather(const float *acc, const int32_t *idx, int64_t m,
                         float *out)
{
    for (int64_t q = 0; q < m; ++q)
        out[q] = acc[idx[q]];
}

void micro_oracle_zero(float *acc, const int32_t *idx, int64_t m)
{
    for (int64_t q = 0; q < m; ++q)
        acc[idx[q]] = 0.0f;
}

int micro_oracle_update(float *x, const int32_t *idx, const float *sums,
                        int64_t m, int32_t world)
{
    if (world < 1)
        return -1;
    float n = (float)world;
    for (int64_t q = 0; q < m; ++q) {
        float average = sums[q] / n;
        x[idx[q]] = x[idx[q]] - average;
    }
    return 0;
}

/* Sec. 2: the local error is the vector of accumulated, not yet selected
 * gradients; its L2 norm is the paper's per-worker error (Eq. 1 averages it
 * over the workers).  This returns the squared norm over one range. */
double micro_oracle_sumsq(const float *residual, int64_t start, int64_t len)
{
    double sum = 0.0;
    for (int64_t j = start; j < start + len; ++j) {
        double v = (double)residual[j];
        sum = sum + v * v;
    }
    return sum;
}

int micro_oracle_sweep(const float *grad, float *residual, int64_t n_total,
                       int32_t world, double density,
                       const micro_oracle_rule *rule, double *theta,
                       int32_t *out_idx, float *out_val, int64_t *k,
                       double *sumsq)
{
    if (grad == NULL || residual == NULL || rule == NULL || theta == NULL ||
        k == NULL || world < 1 || n_total < 0)
        return -1;
    if (!(density > 0.0 && density <= 1.0))
        return -1;
    for (int32_t r = 0; r < world; ++r)
        if (!(theta[r] > 0.0) || isinf(theta[r]))
            return -1;
    if (n_total > 0 && (out_idx == NULL || out_val == NULL))
        return -1;
    int64_t written = 0;
    for (int32_t r = 0; r < world; ++r) {
        int64_t start = 0, len = 0;
        micro_oracle_partition(n_total, r, world, &start, &len);
        int64_t kr = micro_oracle_select(grad, residual, start, len, theta[r],
                                         out_idx + written, out_val + written);
        theta[r] = micro_oracle_estimate(rule, density, len, kr, theta[r]);
        k[r] = kr;
        written = written + kr;
        if (sumsq != NULL)
            sumsq[r] = micro_oracle_sumsq(residual, start, len);
    }
    return 0;
}

/* Sec. 1 and its density footnote: a sorting-based sparsifier orders all
 * values and keeps the k largest; the values here are the error-feedback
 * accumulations of Sec. 2, ordered by magnitude.  Readings where the paper
 * says nothing: equal magnitudes are ordered by index (the lower index ranks
 * higher), and a NaN is never selected, as under the threshold rule, whose
 * compare is false for NaN.  Written as the definition: accumulate, sort,
 * take the first k, then emit in index order. */
typedef struct oracle_ranked {
    float mag;
    int64_t idx;
} oracle_ranked;

static int larger_magnitude_first(const void *pa, const void *pb)
{
    const oracle_ranked *a = (const oracle_ranked *)pa;
    const oracle_ranked *b = (const oracle_ranked *)pb;
    if (a->mag > b->mag)
        return -1;
    if (a->mag < b->mag)
        return 1;
    if (a->idx < b->idx)
        return -1;
    if (a->idx > b->idx)
        return 1;
    return 0;
}

int64_t micro_oracle_topk_count(double density, int64_t len)
{
    if (len <= 0)
        return 0;
    double f = floor(density * (double)len);
    int64_t k = (int64_t)f;
    if (k < 1)
        k = 1;
    if (k > len)
        k = len;
    return k;
}

int micro_oracle_topk_select(const float *grad, float *residual, int64_t start,
                             int64_t len, double density, int32_t *out_idx,
                             float *out_val, int64_t *k_out, double *kth)
{
    if (grad == NULL || residual == NULL || k_out == NULL || kth == NULL ||
        start < 0 || len < 0)
        return -1;
    if (!(density > 0.0 && density <= 1.0))
        return -1;
    if (len > 0 && (out_idx == NULL || out_val == NULL))
        return -1;
    size_t n = (size_t)len;
    float *acc = (float *)malloc((n > 0 ? n : 1) * sizeof(float));
    oracle_ranked *ranked =
        (oracle_ranked *)malloc((n > 0 ? n : 1) * sizeof(oracle_ranked));
    unsigned char *chosen = (unsigned char *)calloc(n > 0 ? n : 1, 1);
    if (acc == NULL || ranked == NULL || chosen == NULL) {
        free(acc);
        free(ranked);
        free(chosen);
        return -1;
    }
    size_t valid = 0;
    for (size_t i = 0; i < n; ++i) {
        acc[i] = grad[start + (int64_t)i] + residual[start + (int64_t)i];
        if (!isnan(acc[i])) {
            ranked[valid].mag = fabsf(acc[i]);
            ranked[valid].idx = start + (int64_t)i;
            valid = valid + 1;
        }
    }
    qsort(ranked, valid, sizeof(oracle_ranked), larger_magnitude_first);
    int64_t want = micro_oracle_topk_count(density, len);
    int64_t take = want < (int64_t)valid ? want : (int64_t)valid;
    for (int64_t r = 0; r < take; ++r)
        chosen[ranked[r].idx - start] = 1;
    if (take > 0)
        *kth = (double)ranked[take - 1].mag;
    int64_t k = 0;
    for (size_t i = 0; i < n; ++i) {
        int64_t j = start + (int64_t)i;
        if (chosen[i]) {
            out_idx[k] = (int32_t)j;
            out_val[k] = acc[i];
            k = k + 1;
            residual[j] = 0.0f;
        } else {
            residual[j] = acc[i];
        }
    }
    *k_out = k;
    free(acc);
    free(ranked);
    free(chosen);
    return 0;
}
