// Drives the host library's device-free entry points under AddressSanitizer
// and UndefinedBehaviorSanitizer (built for the host only and run by
// tests/test_host_sanitize.py on a machine without a GPU): the partition and
// cycle helpers, the threshold update and its binary32 form, status strings,
// init's argument errors and its failure without a device, and every entry
// point handed a NULL context.  Prints "ok" and exits 0 when every check
// holds.
#include <cfloat>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>

#include "micro_sparsify.h"

static int failures = 0;

#define CHECK(cond)                                                     \
    do {                                                                \
        if (!(cond)) {                                                  \
            std::fprintf(stderr, "FAILED line %d: %s\n", __LINE__, #cond); \
            ++failures;                                                 \
        }                                                               \
    } while (0)

int main() {
    // partition: tiles [0, n) for every world, balanced, rejects bad input
    for (int64_t n : {0LL, 1LL, 2LL, 7LL, 1000LL, 2147483647LL}) {
        for (int32_t world : {1, 2, 3, 7, 64, 1000}) {
            int64_t next = 0;
            for (int32_t r = 0; r < world; ++r) {
                int64_t s = -1, len = -1;
                CHECK(micro_partition(n, r, world, &s, &len) == MICRO_OK);
                CHECK(s == next && len >= 0);
                CHECK(len == n / world || len == n / world + 1);
                next = s + len;
            }
            CHECK(next == n);
            int64_t s = -5, len = -5;
            CHECK(micro_partition(n, world, world, &s, &len) == MICRO_EINVAL);
            CHECK(micro_partition(n, -1, world, &s, &len) == MICRO_EINVAL);
            CHECK(s == -5 && len == -5);
        }
    }
    int64_t s0, l0;
    CHECK(micro_partition(-1, 0, 1, &s0, &l0) == MICRO_EINVAL);
    CHECK(micro_partition(10, 0, 0, &s0, &l0) == MICRO_EINVAL);
    CHECK(micro_partition(10, 0, 1, nullptr, &l0) == MICRO_EINVAL);

    // cycle: a permutation of the partitions at every iteration
    for (int32_t world : {1, 2, 5, 16}) {
        for (int64_t t : {0LL, 1LL, 17LL, 1000000007LL}) {
            unsigned seen = 0;
            for (int32_t w = 0; w < world; ++w) {
                int32_t c = -1;
                CHECK(micro_cycle(t, w, world, &c) == MICRO_OK);
                CHECK(c >= 0 && c < world);
                if (c >= 0 && c < 32) seen |= 1u << c;
            }
            CHECK(seen == (world >= 32 ? ~0u : (1u << world) - 1u));
        }
    }
    int32_t c0;
    CHECK(micro_cycle(-1, 0, 4, &c0) == MICRO_EINVAL);
    CHECK(micro_cycle(0, 4, 4, &c0) == MICRO_EINVAL);
    CHECK(micro_cycle(0, 0, 0, &c0) == MICRO_EINVAL);
    CHECK(micro_cycle(0, 0, 4, nullptr) == MICRO_EINVAL);

    // threshold update: direction, fixed point, empty partition, bad input
    micro_config cfg;
    micro_config_default(&cfg);
    for (const micro_config* c : {static_cast<const micro_config*>(nullptr), static_cast<const micro_config*>(&cfg)}) {
        double th = 2.0;
        CHECK(micro_estimate_threshold(c, 0.01, 100000, 5000, &th) == MICRO_OK && th > 2.0);
        th = 2.0;
        CHECK(micro_estimate_threshold(c, 0.01, 100000, 10, &th) == MICRO_OK && th < 2.0);
        th = 2.0;
        CHECK(micro_estimate_threshold(c, 0.01, 100000, 1000, &th) == MICRO_OK && th == 2.0);
        th = 2.0;
        CHECK(micro_estimate_threshold(c, 0.01, 0, 0, &th) == MICRO_OK && th == 2.0);
        CHECK(micro_estimate_threshold(c, 0.0, 100, 1, &th) == MICRO_EINVAL);
        CHECK(micro_estimate_threshold(c, std::nan(""), 100, 1, &th) == MICRO_EINVAL);
        CHECK(micro_estimate_threshold(c, 0.5, 100, 101, &th) == MICRO_EINVAL);
        CHECK(micro_estimate_threshold(c, 0.5, -1, 0, &th) == MICRO_EINVAL);
        CHECK(micro_estimate_threshold(c, 0.5, 100, 1, nullptr) == MICRO_EINVAL);
    }

    // the comparators: hard threshold keeps theta; the top-k threshold comes
    // from the values, so the host-only update and the allocation-free step
    // refuse that rule before any device work
    {
        micro_config hard = cfg, topk = cfg;
        hard.rule = MICRO_RULE_HARD_THRESHOLD;
        topk.rule = MICRO_RULE_TOPK;
        double th = 2.0;
        CHECK(micro_estimate_threshold(&hard, 0.01, 100000, 5000, &th) == MICRO_OK && th == 2.0);
        CHECK(micro_estimate_threshold(&topk, 0.01, 100000, 5000, &th) == MICRO_EINVAL && th == 2.0);
        float gg[8] = {1, 2, 3, 4, 5, 6, 7, 8}, rr[8] = {0}, vv[8];
        int32_t ii[8];
        int64_t kk = -4;
        CHECK(micro_sparsify_step_noalloc(gg, rr, 8, 0, 1, 0.5, &th, ii, vv, &kk, nullptr, &topk) == MICRO_EINVAL);
        CHECK(kk == -4 && th == 2.0 && rr[0] == 0.0f);
        micro_config unknown = cfg;
        unknown.rule = 4;
        CHECK(micro_estimate_threshold(&unknown, 0.01, 100000, 5000, &th) == MICRO_EINVAL);
    }

    // binary32 threshold: the smallest float not below theta
    for (double th : {1e-45, 1e-40, 0.1, 1.0, 2.33, 3.4028234663852886e38, 1e300}) {
        float f = -1.0f;
        CHECK(micro_threshold_f32(th, &f) == MICRO_OK);
        CHECK(static_cast<double>(f) >= th);
        if (std::isfinite(f)) CHECK(static_cast<double>(std::nextafter(f, 0.0f)) < th);
    }
    float f0;
    CHECK(micro_threshold_f32(0.0, &f0) == MICRO_EINVAL);
    CHECK(micro_threshold_f32(-1.0, &f0) == MICRO_EINVAL);
    CHECK(micro_threshold_f32(std::numeric_limits<double>::infinity(), &f0) == MICRO_EINVAL);
    CHECK(micro_threshold_f32(1.0, nullptr) == MICRO_EINVAL);

    // status strings, including a code that does not exist
    for (int st = 0; st <= 6; ++st) {
        const char* name = micro_status_string(static_cast<micro_status>(st));
        CHECK(name != nullptr && std::strlen(name) > 0);
    }

    // init: argument errors, then no device
    micro_ctx* ctx = reinterpret_cast<micro_ctx*>(0x1);
    CHECK(micro_sparsify_init(nullptr, 10, nullptr, nullptr) == MICRO_EINVAL);
    CHECK(micro_sparsify_init(&ctx, -1, nullptr, nullptr) == MICRO_EINVAL && ctx == nullptr);
    ctx = reinterpret_cast<micro_ctx*>(0x1);
    CHECK(micro_sparsify_init(&ctx, 2147483648LL, nullptr, nullptr) == MICRO_ERANGE && ctx == nullptr);
    micro_config bad = cfg;
    bad.variant = 99;
    CHECK(micro_sparsify_init(&ctx, 10, nullptr, &bad) == MICRO_EINVAL && ctx == nullptr);
    bad = cfg;
    bad.lo = -1.0;
    CHECK(micro_sparsify_init(&ctx, 10, nullptr, &bad) == MICRO_EINVAL && ctx == nullptr);
    const micro_status st = micro_sparsify_init(&ctx, 1000, nullptr, &cfg);
    CHECK(st == MICRO_EHIP && ctx == nullptr);
    CHECK(std::strlen(micro_last_error(nullptr)) > 0);

    // every context entry point rejects a NULL context without touching anything
    float g[4] = {1, 2, 3, 4}, r[4] = {0, 0, 0, 0}, v[4];
    int32_t idx[4];
    double th = 1.0;
    int64_t k = -3;
    CHECK(micro_sparsify_step(nullptr, g, r, 0, 1, 0.5, &th, idx, v, &k) == MICRO_EINVAL);
    CHECK(k == -3 && th == 1.0 && r[0] == 0.0f);
    micro_step_stats stats;
    CHECK(micro_sparsify_last_stats(nullptr, &stats) == MICRO_EINVAL);
    CHECK(std::strlen(micro_last_error(nullptr)) > 0);
    micro_sparsify_free(nullptr);

    if (failures != 0) return 1;
    std::printf("ok\n");
    return 0;
}
