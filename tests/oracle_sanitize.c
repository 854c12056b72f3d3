/*
 * Drives every function of the CPU oracle over edge cases under AddressSanitizer
 * and UndefinedBehaviorSanitizer (built and run by tests/test_oracle_sanitize.py).
 * Buffers are allocated at exactly the sizes the oracle's contracts state, so a
 * read or write one element past them is reported.  The driver also checks the
 * conservation and ordering invariants of each result, so a wrong answer fails
 * too.  Exit status 0 and the line "ok" mean that every case passed.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "micro_oracle.h"

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;

static uint32_t next_u32(void) { /* xorshift64* */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (uint32_t)((rng_state * 0x2545f4914f6cdd1dull) >> 32);
}

static float next_value(int regime) {
    const float u = (float)((next_u32() >> 8) + 1) / 16777217.0f; /* (0, 1) */
    float v = (u - 0.5f) * 8.0f;
    switch (regime) {
        case 1: /* specials mixed in */
            switch (next_u32() % 16) {
                case 0: return NAN;
                case 1: return INFINITY;
                case 2: return -INFINITY;
                case 3: return -0.0f;
                case 4: return 1e-40f; /* subnormal */
                default: return v;
            }
        case 2: return v * 1e-30f; /* nothing reaches the threshold */
        default: return v;
    }
}

static void *alloc(size_t n, size_t size) { /* zero elements: still a distinct allocation */
    void *p = malloc(n * size + (n == 0));
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    return p;
}

static int fail(const char *what, int64_t n, int32_t world) {
    fprintf(stderr, "FAILED: %s (n=%lld world=%d)\n", what, (long long)n, world);
    return 1;
}

/* Conservation (selected: value = acc, residual = +0; else residual = acc),
 * ordering and range of one partition's result. */
static int check_partition(const float *g, const float *res0, const float *res1, int64_t s, int64_t len,
                           double theta, const int32_t *idx, const float *val, int64_t k) {
    int64_t q = 0;
    for (int64_t j = s; j < s + len; ++j) {
        const float acc = g[j] + res0[j];
        const int sel = fabs((double)acc) >= theta;
        if (sel) {
            if (q >= k || idx[q] != j || memcmp(&val[q], &acc, 4) != 0) return 0;
            if (res1[j] != 0.0f || signbit(res1[j])) return 0;
            ++q;
        } else if (memcmp(&res1[j], &acc, 4) != 0) {
            return 0;
        }
    }
    return q == k;
}

static int res1_nonzero(float v) { return v != 0.0f || signbit(v); }

static int run_case(int64_t n, int32_t world, int regime, double theta) {
    micro_oracle_rule rule;
    micro_oracle_default_rule(&rule);
    float *g = alloc((size_t)n, sizeof(float));
    float *res = alloc((size_t)n, sizeof(float));
    float *res0 = alloc((size_t)n, sizeof(float));
    for (int64_t j = 0; j < n; ++j) {
        g[j] = next_value(regime);
        res[j] = next_value(regime) * 0.5f;
    }
    int bad = 0;

    /* every partition on its own, outputs sized to the partition */
    for (int32_t r = 0; r < world && !bad; ++r) {
        int64_t s, len, k;
        if (micro_oracle_partition(n, r, world, &s, &len) != 0) return fail("partition", n, world);
        int32_t *idx = alloc((size_t)len, sizeof(int32_t));
        float *val = alloc((size_t)len, sizeof(float));
        memcpy(res0, res, (size_t)n * sizeof(float));
        double th = theta;
        if (micro_oracle_step(g, res, n, r, world, 0.01, &rule, &th, idx, val, &k) != 0)
            bad = fail("step", n, world);
        else if (!check_partition(g, res0, res, s, len, theta, idx, val, k))
            bad = fail("step invariants", n, world);
        const double sq = micro_oracle_sumsq(res, s, len);
        if (!(sq >= 0.0) && !isnan(sq)) bad = fail("sumsq sign", n, world);
        free(idx);
        free(val);
    }

    /* a full error-feedback pass of every worker at a few iterations */
    for (int64_t t = 0; t < 3 && !bad; ++t) {
        for (int32_t w = 0; w < world && !bad; ++w) {
            const int32_t c = micro_oracle_cycle(t, w, world);
            int64_t s, len, k;
            int32_t cyc;
            if (c < 0 || micro_oracle_partition(n, c, world, &s, &len) != 0) return fail("cycle", n, world);
            int32_t *idx = alloc((size_t)len, sizeof(int32_t));
            float *val = alloc((size_t)len, sizeof(float));
            memcpy(res0, res, (size_t)n * sizeof(float));
            double th = theta;
            if (micro_oracle_ef_step(g, res, n, t, w, world, 0.01, &rule, &th, idx, val, &k, &cyc) != 0 ||
                cyc != c)
                bad = fail("ef_step", n, world);
            else if (!check_partition(g, res0, res, s, len, theta, idx, val, k))
                bad = fail("ef_step invariants", n, world);
            free(idx);
            free(val);
        }
    }

    /* the sweep of all partitions, outputs sized to the vector */
    if (!bad) {
        int32_t *idx = alloc((size_t)n, sizeof(int32_t));
        float *val = alloc((size_t)n, sizeof(float));
        double *th = alloc((size_t)world, sizeof(double));
        int64_t *k = alloc((size_t)world, sizeof(int64_t));
        double *sq = alloc((size_t)world, sizeof(double));
        for (int32_t r = 0; r < world; ++r) th[r] = theta * (1.0 + 0.01 * r);
        if (micro_oracle_sweep(g, res, n, world, 0.01, &rule, th, idx, val, k, sq) != 0)
            bad = fail("sweep", n, world);
        int64_t total = 0;
        for (int32_t r = 0; r < world && !bad; ++r) total += k[r];
        for (int64_t q = 1; q < total && !bad; ++q)
            if (idx[q] <= idx[q - 1]) bad = fail("sweep order", n, world);
        free(idx);
        free(val);
        free(th);
        free(k);
        free(sq);
    }

    /* accumulate, then gather / zero / update at a sorted union of indices */
    if (!bad) {
        float *acc = alloc((size_t)n, sizeof(float));
        micro_oracle_accumulate(g, res, n, acc);
        int64_t m = 0;
        int32_t *u = alloc((size_t)n, sizeof(int32_t));
        for (int64_t j = 0; j < n; ++j)
            if (next_u32() % 7 == 0) u[m++] = (int32_t)j;
        float *out = alloc((size_t)m, sizeof(float));
        float *x = alloc((size_t)n, sizeof(float));
        for (int64_t j = 0; j < n; ++j) x[j] = next_value(0);
        micro_oracle_gather(acc, u, m, out);
        micro_oracle_zero(acc, u, m);
        for (int64_t q = 0; q < m && !bad; ++q)
            if (acc[u[q]] != 0.0f) bad = fail("zero", n, world);
        if (micro_oracle_update(x, u, out, m, world) != 0) bad = fail("update", n, world);
        free(acc);
        free(u);
        free(out);
        free(x);
    }

    /* the exact top-k comparator on every partition, outputs sized to it */
    static const double densities[] = {1e-9, 0.01, 0.5, 1.0};
    for (size_t di = 0; di < sizeof densities / sizeof *densities && !bad; ++di) {
        for (int32_t r = 0; r < world && !bad; ++r) {
            int64_t s, len, k;
            micro_oracle_partition(n, r, world, &s, &len);
            int32_t *idx = alloc((size_t)len, sizeof(int32_t));
            float *val = alloc((size_t)len, sizeof(float));
            memcpy(res0, res, (size_t)n * sizeof(float));
            double kth = -1.0;
            if (micro_oracle_topk_select(g, res, s, len, densities[di], idx, val, &k, &kth) != 0) {
                bad = fail("topk_select", n, world);
            } else {
                /* the count, the order, conservation, and every selected
                 * magnitude at least every other value's that is not NaN */
                int64_t valid = 0;
                for (int64_t j = s; j < s + len; ++j) valid += !isnan(g[j] + res0[j]);
                const int64_t want = micro_oracle_topk_count(densities[di], len);
                if (k != (want < valid ? want : valid)) bad = fail("topk count", n, world);
                if (!bad && k > 0 && !check_partition(g, res0, res, s, len, kth, idx, val, k)) {
                    /* equal magnitudes at the k-th may stay: check by selection flags instead */
                    int64_t q = 0;
                    for (int64_t j = s; j < s + len && !bad; ++j) {
                        const float acc = g[j] + res0[j];
                        const int sel = q < k && idx[q] == j;
                        if (sel) {
                            if (memcmp(&val[q], &acc, 4) != 0 || res1_nonzero(res[j])) bad = fail("topk selected", n, world);
                            if (!(fabs((double)acc) >= kth)) bad = fail("topk below kth", n, world);
                            ++q;
                        } else {
                            if (memcmp(&res[j], &acc, 4) != 0) bad = fail("topk residual", n, world);
                            if (!isnan(acc) && fabs((double)acc) > kth) bad = fail("topk above kth left", n, world);
                        }
                    }
                    if (!bad && q != k) bad = fail("topk order", n, world);
                }
                if (!bad && k == 0 && kth != -1.0) bad = fail("topk kth untouched", n, world);
            }
            free(idx);
            free(val);
        }
    }
    if (!bad) {
        int64_t k = -5;
        double kth = 3.0;
        if (micro_oracle_topk_select(g, res, 0, n, 0.0, NULL, NULL, &k, &kth) != -1 || k != -5 || kth != 3.0)
            bad = fail("topk_select rejects density 0", n, world);
        if (micro_oracle_topk_count(0.5, 0) != 0) bad = fail("topk_count of nothing", n, world);
    }

    /* invalid arguments write nothing */
    if (!bad) {
        int64_t s = -7, len = -7;
        if (micro_oracle_partition(n, world, world, &s, &len) != -1 || s != -7 || len != -7)
            bad = fail("partition rejects rank == world", n, world);
        if (micro_oracle_cycle(-1, 0, world) != -1) bad = fail("cycle rejects t < 0", n, world);
    }

    free(g);
    free(res);
    free(res0);
    return bad;
}

int main(void) {
    static const int64_t sizes[] = {0, 1, 2, 3, 5, 17, 64, 1000, 4097, 65537};
    static const int32_t worlds[] = {1, 2, 3, 7, 16, 64};
    static const double thetas[] = {1e-30, 0.5, 2.0, 1e30};
    int bad = 0;
    for (size_t a = 0; a < sizeof sizes / sizeof *sizes; ++a)
        for (size_t b = 0; b < sizeof worlds / sizeof *worlds; ++b)
            for (int regime = 0; regime < 3; ++regime)
                for (size_t c = 0; c < sizeof thetas / sizeof *thetas; ++c)
                    bad |= run_case(sizes[a], worlds[b], regime, thetas[c]);
    if (bad) return 1;
    printf("ok\n");
    return 0;
}
