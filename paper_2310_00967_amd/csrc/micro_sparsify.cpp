// Host side of the C ABI declared in include/micro_sparsify.h: argument
// validation, the Sec. 4.1 partition, the binary32 form of the threshold,
// kernel launch, the selected-count readback and the Sec. 4.3 threshold
// update in binary64.  Compiled with -ffp-contract=off.
#include "micro_sparsify.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <limits>
#include <mutex>
#include <new>
#include <string>

#include "sparsify_kernel.h"
#include "static_scratch.h"
#include "topk_kernel.h"

struct micro_ctx {
    int device = -1;
    int compute_units = 256;                 // of the device, read at init
    int64_t n_total = 0;
    hipStream_t stream = nullptr;
    micro_config cfg{};
    bool has_staged = true;                  // scratch of the staged schedule allocated
    bool has_ticket = false;                 // scratch of the ticket schedule allocated
    int64_t tile_capacity = 0;               // staged tiles of the largest partition (or sweep)
    int64_t ticket_capacity = 0;             // ticket tiles of the largest partition
    // staged schedule: tile counts, staged pairs, chunk look-back words
    uint32_t* d_tile_counts = nullptr;
    uint32_t* d_tile_excl = nullptr;
    uint32_t* d_flagged_list = nullptr;
    uint32_t* d_split_tile = nullptr;
    double* d_tile_sumsq = nullptr;          // sweep: per tile
    int64_t split_capacity = 0;
    uint2* d_stage = nullptr;                // (index, value bits) pairs
    uint64_t* d_chunk_status = nullptr;
    int64_t chunk_capacity = 0;
    uint64_t* d_tile_words = nullptr;        // fused schedule: epoch-tagged tile counts
    // ticket schedule: tile look-back words
    uint64_t* d_status = nullptr;
    unsigned long long* d_tickets = nullptr; // [0] tile ticket of the one-pass schedule
    int64_t* d_count = nullptr;              // [0] selected count, [1] (epoch << 32) | flagged tiles
    int64_t* h_count = nullptr;              // mapped pinned host memory stored by the kernels: [0] k,
                                             // [1] redone tiles, [2 + r] a sweep's counts
    int64_t* h_count_dev = nullptr;          // the device's address of h_count
    double* h_sumsq = nullptr;               // mapped pinned host memory: a sweep's squared norms, per chunk
    double* h_sumsq_dev = nullptr;
    // top-k comparator: radix-select counters and state, and its result for the host
    uint32_t* d_topk = nullptr;              // kTopkBins counters (zero between passes), kTopkStateWords
    int64_t* h_topk = nullptr;               // mapped pinned host memory, kTopkHostWords
    int64_t* h_topk_dev = nullptr;
    uint32_t epoch = 0;                      // epoch of the last launch
    bool needs_reset = false;                // scratch state unknown after a failure
    hipEvent_t ev[2] = {nullptr, nullptr};
    micro_step_stats stats{};
    std::string last_error;
};

namespace {

// Makes the context's device current for the scope of a call and restores the
// caller's current device afterwards, so a context works whatever device the
// calling thread has selected since init.
struct DeviceScope {
    int previous = -1;
    bool switched = false;
    explicit DeviceScope(int device) {
        if (device >= 0 && hipGetDevice(&previous) == hipSuccess && previous != device)
            switched = hipSetDevice(device) == hipSuccess;
    }
    ~DeviceScope() {
        if (switched) (void)hipSetDevice(previous);
    }
    DeviceScope(const DeviceScope&) = delete;
    DeviceScope& operator=(const DeviceScope&) = delete;
};

// Largest partition that an AUTO context runs on the ticket schedule.  On
// MI355X the ticket schedule's single launch took 8.7 us of device time for
// 262,144 values against 15.6 us for the staged schedule's three, and lost
// from 3.2M values on (27 us against 23 us).
constexpr int64_t kAutoTicketMax = int64_t(1) << 20;

thread_local std::string g_init_error = "no error";

void set_error(micro_ctx* ctx, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (ctx)
        ctx->last_error = buf;
    else
        g_init_error = buf;
}

micro_status hip_fail(micro_ctx* ctx, hipError_t err, const char* what) {
    set_error(ctx, "%s failed: %s", what, hipGetErrorString(err));
    if (ctx) ctx->needs_reset = true;
    return MICRO_EHIP;
}

bool config_valid(const micro_config& c) {
    if (c.rule != MICRO_RULE_PROPORTIONAL && c.rule != MICRO_RULE_FIXED_STEP && c.rule != MICRO_RULE_HARD_THRESHOLD &&
        c.rule != MICRO_RULE_TOPK)
        return false;
    if (!std::isfinite(c.beta) || c.beta < 0.0) return false;
    if (!std::isfinite(c.lo) || !std::isfinite(c.hi) || !(c.lo > 0.0) || !(c.hi >= c.lo)) return false;
    if (!std::isfinite(c.alpha) || c.alpha < 0.0 || !(c.alpha < 1.0)) return false;
    if (c.variant != MICRO_VARIANT_AUTO && c.variant != MICRO_VARIANT_TICKET &&
        c.variant != MICRO_VARIANT_STAGED)
        return false;
    if ((c.flags & ~(MICRO_FLAG_TIME_KERNEL | MICRO_FLAG_SEPARATE_SCAN)) != 0) return false;
    return true;
}

bool density_valid(double d) { return d > 0.0 && d <= 1.0; }

bool theta_valid(double t) { return std::isfinite(t) && t > 0.0; }

// Sec. 4.3 threshold scaling (the reading of the paper's Estimate): the
// target count is d * P; the proportional rule multiplies the threshold by
// 1 + beta * (k - target) / target clamped to [lo, hi]; the fixed-step rule
// by 1 + alpha or 1 - alpha according to the sign of k - target.  Each
// operation is one IEEE binary64 rounding, in this order.  The
// hard-threshold comparator keeps the threshold as it is.  (The top-k
// comparator's threshold comes from the values: execute_step sets it.)
double next_threshold(const micro_config& c, double density, int64_t part_len, int64_t k,
                      double theta) {
    if (part_len == 0 || c.rule == MICRO_RULE_HARD_THRESHOLD || c.rule == MICRO_RULE_TOPK) return theta;
    const double target = density * static_cast<double>(part_len);
    const double got = static_cast<double>(k);
    if (c.rule == MICRO_RULE_FIXED_STEP) {
        if (got > target) return theta * (1.0 + c.alpha);
        if (got < target) return theta * (1.0 - c.alpha);
        return theta;
    }
    const double relative_error = (got - target) / target;
    const double gain = c.beta * relative_error;
    double factor = 1.0 + gain;
    if (factor < c.lo) factor = c.lo;
    if (factor > c.hi) factor = c.hi;
    return theta * factor;
}

float threshold_as_f32(double theta) {
    float f = static_cast<float>(theta);  // round to nearest
    if (static_cast<double>(f) < theta) f = std::nextafter(f, std::numeric_limits<float>::infinity());
    return f;
}

bool ranges_overlap(const void* a, size_t an, const void* b, size_t bn) {
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + bn && b0 < a0 + an;
}

micro_status reset_scratch(micro_ctx* ctx) {
    hipError_t e = hipMemsetAsync(ctx->d_tickets, 0, sizeof(unsigned long long), ctx->stream);
    if (e == hipSuccess) e = hipMemsetAsync(ctx->d_count, 0, 2 * sizeof(int64_t), ctx->stream);
    if (e == hipSuccess && ctx->d_status)
        e = hipMemsetAsync(ctx->d_status, 0, sizeof(uint64_t) * ctx->ticket_capacity, ctx->stream);
    if (e == hipSuccess && ctx->d_chunk_status)
        e = hipMemsetAsync(ctx->d_chunk_status, 0, sizeof(uint64_t) * ctx->chunk_capacity, ctx->stream);
    if (e == hipSuccess && ctx->d_tile_words)
        e = hipMemsetAsync(ctx->d_tile_words, 0, sizeof(uint64_t) * ctx->tile_capacity, ctx->stream);
    if (e == hipSuccess && ctx->d_topk)
        e = hipMemsetAsync(ctx->d_topk, 0, sizeof(uint32_t) * (micro::kTopkBins + micro::kTopkStateWords),
                           ctx->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "scratch reset");
    ctx->epoch = 0;
    ctx->needs_reset = false;
    return MICRO_OK;
}

void release(micro_ctx* ctx) {
    if (!ctx) return;
    DeviceScope scope(ctx->device);
    if (ctx->device >= 0) (void)hipStreamSynchronize(ctx->stream);
    for (hipEvent_t ev : ctx->ev)
        if (ev) (void)hipEventDestroy(ev);
    void* device_buffers[] = {ctx->d_tile_counts, ctx->d_tile_excl, ctx->d_flagged_list, ctx->d_split_tile, ctx->d_tile_sumsq, ctx->d_stage,
                              ctx->d_chunk_status, ctx->d_tile_words, ctx->d_status, ctx->d_tickets,
                              ctx->d_count, ctx->d_topk};
    for (void* p : device_buffers)
        if (p) (void)hipFree(p);
    if (ctx->h_count) (void)hipHostFree(ctx->h_count);
    if (ctx->h_sumsq) (void)hipHostFree(ctx->h_sumsq);
    if (ctx->h_topk) (void)hipHostFree(ctx->h_topk);
    delete ctx;
}


// Workgroups of the move kernel: one per move piece of a count of len, at
// most kMoveGrid, at least min_blocks.  Its grid-stride loops are correct for
// any grid: a larger count only gives each workgroup more pieces.
uint32_t move_grid(int64_t tiles, int64_t len, int64_t span, int64_t min_blocks) {
    int64_t blocks = (tiles + len + span - 1) / span;
    if (blocks > micro::kMoveGrid) blocks = micro::kMoveGrid;
    if (blocks < min_blocks) blocks = min_blocks;
    return static_cast<uint32_t>(blocks < 1 ? 1 : blocks);
}

// Items per move piece.  The merged sequence holds one item per tile and one
// per selected value, about tiles + density * values of them.  A long
// sequence (at least two kMoveSpan-item pieces per compute unit) takes
// kMoveSpan-item pieces, a short loop per workgroup; a shorter one, whose
// step is bound by the move kernel's round trips rather than its bytes,
// takes smaller pieces, which put more workgroups to work and give each
// less to copy after its last load: kMoveSpanSmall down to one such piece
// per compute unit, kMoveSpanTiny below.  Measured (five runs each, same
// box): BERT-large rank 3 (41.9M values, d = 0.01, about 460,000 items)
// 70.6%, 71.4% and 71.2% of 8 TB/s with 2048-, 1024- and 512-item pieces;
// ResNet-50 rank 0 (3.2M values, d = 0.001, about 6,300 items) 26.5%, 27.0%
// and 27.3%; the GPT-1.3B partition's move kernel took 53 us with 4096-item
// pieces and 78 us with 2048 (an earlier build of the kernel).
// Largest sweep, in scan chunks of a million values, whose stream and scan
// passes run as one launch.  Measured on MI355X (device time per sweep, fused
// against separate, same box): ResNet-18's 16 partitions (16 chunks) 43.6
// against 46.9 us, ResNet-50's 8 (32 chunks) 72.4-73.2 against 72.2 us,
// BERT-large's 8 (320 chunks) 665-667 against 655-657 us.
constexpr int64_t kFusedSweepMaxChunks = 64;

uint32_t move_span_for(const micro_ctx* ctx, int64_t tiles, double expected_pairs) {
    const double items = static_cast<double>(tiles) + expected_pairs;
    if (items >= 2.0 * ctx->compute_units * micro::kMoveSpan) return micro::kMoveSpan;
    if (items >= 1.0 * ctx->compute_units * micro::kMoveSpanSmall) return micro::kMoveSpanSmall;
    return micro::kMoveSpanTiny;
}

bool misaligned4(std::initializer_list<const void*> ptrs) {
    uintptr_t bits = 0;
    for (const void* p : ptrs) bits |= reinterpret_cast<uintptr_t>(p);
    return (bits & 3u) != 0;
}

micro_status run_segments(micro_ctx* ctx, const float* grad, float* residual, int32_t count, const int64_t* starts,
                          const int64_t* lens, const float* threshold_f, double expected_pairs, int32_t* out_idx,
                          float* out_val, int64_t* k, double* sumsq);

// Arguments of a step over [start, start + len) of a vector of n_total values
// (whole_vector: grad and residual are accessed over all of it): NULL
// pointers, density, threshold (unless the rule does not use it), alignment
// and overlapping ranges.  The message goes to ctx, or to the calling
// thread's error when ctx is NULL.
micro_status check_step_args(micro_ctx* ctx, const float* grad, const float* residual, int64_t n_total,
                             int64_t start, int64_t len, bool whole_vector, double density, const double* theta,
                             const int32_t* out_idx, const float* out_val, const int64_t* k,
                             bool threshold_used = true) {
    if (!grad || !residual || !theta || !out_idx || !out_val || !k) {
        set_error(ctx, "NULL pointer argument");
        return MICRO_EINVAL;
    }
    if (!density_valid(density)) {
        set_error(ctx, "density %g outside (0, 1]", density);
        return MICRO_EINVAL;
    }
    if (threshold_used && !theta_valid(*theta)) {
        set_error(ctx, "threshold %g is not finite and positive", *theta);
        return MICRO_EINVAL;
    }
    if (misaligned4({grad, residual, out_idx, out_val})) {
        set_error(ctx, "buffers must be 4-byte aligned");
        return MICRO_EINVAL;
    }
    // the ranges each buffer is accessed over
    const int64_t span_start = whole_vector ? 0 : start;
    const size_t span = static_cast<size_t>(whole_vector ? n_total : len) * sizeof(float);
    const size_t pb = static_cast<size_t>(len) * sizeof(float);
    const void* regions[4] = {grad + span_start, residual + span_start, out_idx, out_val};
    const size_t sizes[4] = {span, span, pb, pb};
    for (int i = 0; i < 4; ++i)
        for (int j = i + 1; j < 4; ++j)
            if (sizes[i] > 0 && sizes[j] > 0 && ranges_overlap(regions[i], sizes[i], regions[j], sizes[j])) {
                set_error(ctx, "grad, residual and output ranges overlap");
                return MICRO_EINVAL;
            }
    return MICRO_OK;
}

// The top-k comparator's k over a partition of len values: Sec. 1's
// density footnote, d = k / n_g, read for a partition: floor(d * len) in
// binary64, at least 1, at most len.
int64_t topk_count(double density, int64_t len) {
    if (len <= 0) return 0;
    int64_t k = static_cast<int64_t>(std::floor(density * static_cast<double>(len)));
    if (k < 1) k = 1;
    if (k > len) k = len;
    return k;
}

float float_from_bits(uint32_t b) {
    float f;
    std::memcpy(&f, &b, sizeof f);
    return f;
}

// How a top-k step runs.  With a usable hint (the incoming theta, normally
// the k-th magnitude the last step returned) the threshold step runs first,
// at 7/8 of the hint rounded down to binary32 (kHint); under the staged
// schedule it sets the residual to +0 only from the hint itself up (rounded
// down to binary32), where the k-th magnitude is expected, so the trim has
// few residual values to change.  When it lists at least k values (and the
// staging pairs hold them), the three histogram passes run over that list and
// the trim cuts it to the top k (kHintList); else the list goes back into the
// residual, which then holds acc over the partition, a first pass runs over
// the residual and either the values from the k-th magnitude's first-digit
// bin up are extracted into the list for the other passes and the trim, or
// (a long list) the passes and the pick run over the residual (kHintPick).
// Without a hint every route starts with the first histogram pass over the
// partition (waited for).  The full route runs the other two passes over the
// partition too (waited for), then the threshold step at the exact k-th
// magnitude, then the trim if values equal to it must be dropped.  The list
// route runs the threshold step at the floor of the first digit's bin
// instead, then the other two passes over the step's output list, then the
// trim; it is taken when that list is at most a quarter of the partition and
// the staging pairs can hold it.  None: every value is NaN, nothing is
// selected.
enum class TopkRoute { kNone, kFull, kList, kHint, kHintList, kHintPick };

struct TopkPlan {
    TopkRoute route = TopkRoute::kNone;
    uint32_t threshold_key = 0;  // the step selects the keys >= this one
    uint32_t zero_key = 0;       // and sets the residual of the keys >= this one to +0
    int64_t kept = 0;            // the values selected in the end: min(k, values not NaN); kHintPick: k
    int64_t listed = 0;          // the entries of the step's output list
    bool trim = false;
};

int32_t topk_route_code(TopkRoute r) {
    switch (r) {
        case TopkRoute::kFull: return MICRO_TOPK_ROUTE_FULL;
        case TopkRoute::kList: return MICRO_TOPK_ROUTE_LIST;
        case TopkRoute::kHintList: return MICRO_TOPK_ROUTE_HINT_LIST;
        case TopkRoute::kHintPick: return MICRO_TOPK_ROUTE_HINT_PICK;
        default: return 0;
    }
}

// The parallel trim's scratch: the staged schedule's staging pairs (free once
// the step's kernels are done), tile counts and tile norms, when they hold a
// list of n entries; else none (the one-workgroup trim).
micro::TopkTrimScratch trim_scratch(const micro_ctx* ctx, int64_t n) {
    micro::TopkTrimScratch t{nullptr, nullptr, nullptr};
    const int64_t chunks = (n + micro::kTopkTrimChunk - 1) / micro::kTopkTrimChunk;
    if (ctx->has_staged && ctx->d_stage && ctx->d_tile_counts && ctx->d_tile_sumsq &&
        n <= ctx->tile_capacity * static_cast<int64_t>(micro::kStageCap) && 2 * chunks <= ctx->tile_capacity)
        t = {ctx->d_stage, ctx->d_tile_counts, ctx->d_tile_sumsq};
    return t;
}

// Workgroups of a histogram pass over n values: enough for the device, at
// most four per compute unit (each thread loops).  Each workgroup adds its
// nonzero counters (up to 2048) to the global ones, so a pass over a short
// list takes fewer workgroups with more values each (kTopkListPerThread).
constexpr int64_t kTopkListPerThread = 16;

uint32_t topk_blocks(const micro_ctx* ctx, int64_t n, int64_t values_per_thread) {
    const int64_t per_block = static_cast<int64_t>(micro::kTopkHistBlock) * values_per_thread;
    const int64_t blocks = std::min<int64_t>((n + per_block - 1) / per_block, 4 * ctx->compute_units);
    return static_cast<uint32_t>(std::max<int64_t>(blocks, 1));
}

// The incoming theta as a hint for this step's k-th magnitude: the step
// first runs at kTopkHintScale times it, rounded down to binary32 (*key: its
// bits).  Taken when theta is positive and finite, the bound a positive
// binary32, k at most an eighth of the partition, and the staged scratch
// there for the trim and the pick.
constexpr double kTopkHintScale = 0.875;

// The largest binary32 at or below x (x >= 0): FLT_MAX above it.
float f32_at_or_below(double x) {
    if (x >= static_cast<double>(std::numeric_limits<float>::max())) return std::numeric_limits<float>::max();
    float f = static_cast<float>(x);
    if (static_cast<double>(f) > x) f = std::nextafter(f, 0.0f);
    return f;
}

bool topk_hint_key(const micro_ctx* ctx, double theta, int64_t k, int64_t len, uint32_t* key) {
    if (!ctx->has_staged || !ctx->d_stage || !ctx->d_tile_counts || !ctx->d_tile_sumsq) return false;
    if (!(theta > 0.0) || !std::isfinite(theta) || k > len / 8) return false;
    const int64_t chunks = (len + micro::kTopkTrimChunk - 1) / micro::kTopkTrimChunk;
    if (2 * chunks > ctx->tile_capacity) return false;
    const double b = theta * kTopkHintScale;
    if (b > static_cast<double>(std::numeric_limits<float>::max())) return false;
    const float f = f32_at_or_below(b);
    if (!(f > 0.0f)) return false;
    std::memcpy(key, &f, sizeof *key);
    return true;
}

micro_status topk_inconsistent(micro_ctx* ctx, const char* where) {
    const volatile int64_t* h = ctx->h_topk;
    set_error(ctx, "top-k select (%s) reported status %lld, key %lld, %lld above, %lld at it, %lld remaining, %lld valid",
              where, static_cast<long long>(h[5]), static_cast<long long>(h[0]), static_cast<long long>(h[1]),
              static_cast<long long>(h[2]), static_cast<long long>(h[3]), static_cast<long long>(h[4]));
    ctx->needs_reset = true;
    return MICRO_EHIP;
}

// The radix select's first pass over acc = grad + residual of
// [start, start + len) and the choice of the route; on the full route also
// its other two passes.  Waits for the device.
micro_status topk_plan(micro_ctx* ctx, const float* grad, const float* residual, int64_t start, int64_t len,
                       double density, bool vec4, TopkPlan* plan) {
    *plan = TopkPlan{};
    micro::TopkArgs t{};
    t.grad = grad;
    t.residual = residual;
    t.start = start;
    t.end = start + len;
    t.vec4 = vec4;
    if (vec4) {  // the 16-byte groups of both vectors (they share the phase)
        const uintptr_t addr = reinterpret_cast<uintptr_t>(grad + start);
        int64_t head = static_cast<int64_t>(((16u - (addr & 15u)) & 15u) / sizeof(float));
        if (head > len) head = len;
        t.body_first = start + head;
        t.body_end = t.body_first + ((t.end - t.body_first) / 4) * 4;
    }
    const int64_t k = topk_count(density, len);
    t.k = static_cast<uint32_t>(k);
    t.words = ctx->d_topk;
    t.host = ctx->h_topk_dev;
    t.blocks = topk_blocks(ctx, len, 8);  // two 16-byte groups a thread
    volatile int64_t* h = ctx->h_topk;
    h[5] = 0;
    hipError_t e = micro::launch_topk_passes(t, micro::TopkSource::kAcc, 0, 0, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "top-k first pass launch");
    if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess) return hip_fail(ctx, e, "hipStreamSynchronize");
    if (h[5] == 2) return MICRO_OK;  // every value is NaN
    const int64_t bin = h[0], greater0 = h[1], in_bin = h[2], remaining = h[3], valid = h[4];
    const int64_t kept = std::min(k, valid);
    const int64_t bin_width = int64_t(1) << micro::kTopkFirstShift;
    if (h[5] != 3 || bin < 0 || bin > micro::kTopkKeyMax || bin % bin_width != 0 || remaining < 1 ||
        remaining > in_bin || greater0 < 0 || greater0 + remaining != kept || greater0 + in_bin > len)
        return topk_inconsistent(ctx, "first pass");
    plan->kept = kept;
    const int64_t listed = greater0 + in_bin;
    if (listed <= len / 4 && trim_scratch(ctx, listed).temp) {
        plan->route = TopkRoute::kList;
        plan->threshold_key = static_cast<uint32_t>(bin);
        plan->zero_key = plan->threshold_key;
        plan->listed = listed;
        plan->trim = true;
        return MICRO_OK;
    }
    h[5] = 0;
    if ((e = micro::launch_topk_passes(t, micro::TopkSource::kAcc, 1, 2, ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "top-k pass launch");
    if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess) return hip_fail(ctx, e, "hipStreamSynchronize");
    const int64_t key = h[0], greater = h[1], equal = h[2], keep = h[3];
    if (h[5] != 1 || key < bin || key >= bin + bin_width || key > micro::kTopkKeyMax || keep < 1 || keep > equal ||
        greater < 0 || greater + keep != kept || greater + equal > len)
        return topk_inconsistent(ctx, "last pass");
    plan->route = TopkRoute::kFull;
    plan->threshold_key = static_cast<uint32_t>(key);
    plan->zero_key = plan->threshold_key;
    plan->listed = greater + equal;
    plan->trim = keep < equal;
    return MICRO_OK;
}

// Enqueued after the step's launches: on the list route the radix select's
// last two passes over the step's output values, then the trim if the plan
// has one.
hipError_t topk_after_step(micro_ctx* ctx, const TopkPlan& plan, int32_t* out_idx, float* out_val, float* residual) {
    hipError_t e = hipSuccess;
    if (plan.route == TopkRoute::kList) {
        micro::TopkArgs t{};
        t.list = out_val;
        t.list_n = plan.listed;
        t.k = static_cast<uint32_t>(plan.kept);  // read by pass 0 only
        t.words = ctx->d_topk;
        t.host = ctx->h_topk_dev;
        t.blocks = topk_blocks(ctx, plan.listed, kTopkListPerThread);
        ctx->h_topk[5] = 0;  // the device last wrote it in the first pass's select, which has been waited for
        if ((e = micro::launch_topk_passes(t, micro::TopkSource::kList, 1, 2, ctx->stream)) != hipSuccess) return e;
    }
    if (plan.trim) {
        const micro::TopkTrimScratch scratch = trim_scratch(ctx, plan.listed);
        e = micro::launch_topk_trim(out_idx, out_val, residual, plan.listed, plan.kept, plan.zero_key, ctx->d_topk,
                                    ctx->h_topk_dev, &scratch, ctx->stream);
    }
    return e;
}

// After the step at the hint's bound listed `listed` values (waited for):
// with at least k of them, and room for the trim, the three passes run over
// that list and the trim cuts it to the top k (enqueued only); else the list
// goes back into the residual, which then holds acc over the partition, and
// the select starts over on it (one more wait).
micro_status topk_after_hint(micro_ctx* ctx, TopkPlan* plan, int64_t listed, float* residual, int64_t start,
                             int64_t len, double density, int32_t* out_idx, float* out_val) {
    const int64_t k = topk_count(density, len);
    micro::TopkArgs t{};
    t.k = static_cast<uint32_t>(k);
    t.words = ctx->d_topk;
    t.host = ctx->h_topk_dev;
    ctx->h_topk[5] = 0;
    plan->listed = listed;
    plan->kept = k;
    hipError_t e;
    if (listed >= k && trim_scratch(ctx, listed).temp) {
        plan->route = TopkRoute::kHintList;
        // with nothing to drop (listed == k) the trim still sets to +0 the
        // residual of kept values the step left at acc (below zero_key)
        plan->trim = listed > k || plan->zero_key > plan->threshold_key;
        t.list = out_val;
        t.list_n = listed;
        t.blocks = topk_blocks(ctx, listed, kTopkListPerThread);
        if ((e = micro::launch_topk_passes(t, micro::TopkSource::kList, 0, 2, ctx->stream)) != hipSuccess)
            return hip_fail(ctx, e, "top-k pass launch");
        if (plan->trim) {
            const micro::TopkTrimScratch scratch = trim_scratch(ctx, listed);
            if ((e = micro::launch_topk_trim(out_idx, out_val, residual, listed, k, plan->zero_key, ctx->d_topk,
                                             ctx->h_topk_dev, &scratch, ctx->stream)) != hipSuccess)
                return hip_fail(ctx, e, "top-k trim launch");
        }
        return MICRO_OK;
    }
    plan->route = TopkRoute::kHintPick;
    plan->trim = false;
    const int64_t chunks = (len + micro::kTopkTrimChunk - 1) / micro::kTopkTrimChunk;
    if (2 * chunks > ctx->tile_capacity) {  // topk_hint_key checked it
        set_error(ctx, "top-k pick needs %lld count words, scratch holds %lld", static_cast<long long>(2 * chunks),
                  static_cast<long long>(ctx->tile_capacity));
        return MICRO_ECAPACITY;
    }
    if ((e = micro::launch_topk_restore(out_idx, out_val, listed, residual, start, start + len, ctx->stream)) !=
        hipSuccess)
        return hip_fail(ctx, e, "top-k restore launch");
    t.residual = residual;
    t.start = start;
    t.end = start + len;
    t.vec4 = true;  // the residual's own 16-byte groups
    const uintptr_t addr = reinterpret_cast<uintptr_t>(residual + start);
    int64_t head = static_cast<int64_t>(((16u - (addr & 15u)) & 15u) / sizeof(float));
    if (head > len) head = len;
    t.body_first = start + head;
    t.body_end = t.body_first + ((t.end - t.body_first) / 4) * 4;
    t.blocks = topk_blocks(ctx, len, 8);
    // The first pass over the residual (waited for) gives the k-th
    // magnitude's first-digit bin.  If everything from the bin's floor up is
    // short, it is extracted into the output list and the other two passes
    // and the trim run over that list; else they and the pick run over the
    // residual.
    volatile int64_t* h = ctx->h_topk;
    if ((e = micro::launch_topk_passes(t, micro::TopkSource::kResidual, 0, 0, ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "top-k pass launch");
    if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess) return hip_fail(ctx, e, "hipStreamSynchronize");
    if (h[5] == 2) return MICRO_OK;  // every value is NaN
    const int64_t bin = h[0], greater0 = h[1], in_bin = h[2], remaining = h[3], valid = h[4];
    const int64_t kept = std::min(k, valid);
    const int64_t bin_width = int64_t(1) << micro::kTopkFirstShift;
    if (h[5] != 3 || bin < 0 || bin > micro::kTopkKeyMax || bin % bin_width != 0 || remaining < 1 ||
        remaining > in_bin || greater0 < 0 || greater0 + remaining != kept || greater0 + in_bin > len)
        return topk_inconsistent(ctx, "first pass over the residual");
    const int64_t extracted = greater0 + in_bin;
    h[5] = 0;
    if (extracted <= len / 4 && trim_scratch(ctx, extracted).temp) {
        if ((e = micro::launch_topk_extract(residual, start, start + len, static_cast<uint32_t>(bin), out_idx, out_val,
                                            ctx->d_tile_counts, ctx->stream)) != hipSuccess)
            return hip_fail(ctx, e, "top-k extract launch");
        micro::TopkArgs l{};
        l.k = static_cast<uint32_t>(k);
        l.words = ctx->d_topk;
        l.host = ctx->h_topk_dev;
        l.list = out_val;
        l.list_n = extracted;
        l.blocks = topk_blocks(ctx, extracted, kTopkListPerThread);
        if ((e = micro::launch_topk_passes(l, micro::TopkSource::kList, 1, 2, ctx->stream)) != hipSuccess)
            return hip_fail(ctx, e, "top-k pass launch");
        // every extracted value had its residual set to +0
        const micro::TopkTrimScratch scratch = trim_scratch(ctx, extracted);
        if ((e = micro::launch_topk_trim(out_idx, out_val, residual, extracted, kept, static_cast<uint32_t>(bin),
                                         ctx->d_topk, ctx->h_topk_dev, &scratch, ctx->stream)) != hipSuccess)
            return hip_fail(ctx, e, "top-k trim launch");
        return MICRO_OK;
    }
    if ((e = micro::launch_topk_passes(t, micro::TopkSource::kResidual, 1, 2, ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "top-k pass launch");
    if ((e = micro::launch_topk_pick(residual, start, start + len, out_idx, out_val, ctx->d_topk, ctx->d_tile_counts,
                                     ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "top-k pick launch");
    return MICRO_OK;
}

// After the wait: the step must have listed what the plan expects; the
// selected count, the k-th magnitude and (returned_sq) the squares of the
// values the trim returned to the residual.
micro_status topk_finish(micro_ctx* ctx, const TopkPlan& plan, int64_t listed_by_step, int64_t* selected,
                         double* theta, double* returned_sq) {
    if (returned_sq) *returned_sq = 0.0;
    const int64_t expected = plan.route == TopkRoute::kNone ? 0 : plan.listed;
    if (listed_by_step != expected) {
        set_error(ctx, "top-k step listed %lld values, the select expected %lld", static_cast<long long>(listed_by_step),
                  static_cast<long long>(expected));
        ctx->needs_reset = true;
        return MICRO_EHIP;
    }
    *selected = 0;
    if (plan.route == TopkRoute::kNone) return MICRO_OK;
    const volatile int64_t* h = ctx->h_topk;
    uint32_t key = plan.threshold_key;
    if (plan.route == TopkRoute::kHintPick) {
        if (h[5] == 2 && plan.listed == 0 && h[4] == 0) return MICRO_OK;  // every value is NaN
        const int64_t k_key = h[0], greater = h[1], equal = h[2], keep = h[3], valid = h[4];
        const int64_t kept = std::min(plan.kept, valid);
        if (h[5] != 1 || k_key < 0 || k_key > micro::kTopkKeyMax || valid < plan.listed || keep < 1 ||
            keep > equal || greater < 0 || greater + keep != kept || greater + equal > valid)
            return topk_inconsistent(ctx, "residual");
        *selected = kept;
        *theta = static_cast<double>(float_from_bits(static_cast<uint32_t>(k_key)));
        return MICRO_OK;
    }
    if (plan.route == TopkRoute::kHintList) {
        const int64_t k_key = h[0], greater = h[1], equal = h[2], keep = h[3];
        if (h[5] != 1 || k_key < plan.threshold_key || k_key > micro::kTopkKeyMax || keep < 1 || keep > equal ||
            greater < 0 || greater + keep != plan.kept || greater + equal > plan.listed)
            return topk_inconsistent(ctx, "hinted list");
        key = static_cast<uint32_t>(k_key);
    }
    if (plan.route == TopkRoute::kList) {
        const int64_t k_key = h[0], greater = h[1], equal = h[2], keep = h[3];
        if (h[5] != 1 || k_key < plan.threshold_key ||
            k_key >= static_cast<int64_t>(plan.threshold_key) + (int64_t(1) << micro::kTopkFirstShift) ||
            k_key > micro::kTopkKeyMax || keep < 1 || keep > equal || greater < 0 || greater + keep != plan.kept ||
            greater + equal > plan.listed)
            return topk_inconsistent(ctx, "output list");
        key = static_cast<uint32_t>(k_key);
    }
    if (plan.trim && returned_sq) {
        const int64_t bits = h[6];
        std::memcpy(returned_sq, &bits, sizeof *returned_sq);
    }
    *selected = plan.kept;
    *theta = static_cast<double>(float_from_bits(key));
    return MICRO_OK;
}

// Validation, launch, count readback and threshold update of one sparsify
// step over [start, start + len); with accumulate_outside the rest of the
// vector is accumulated too (the full error-feedback pass), and with sumsq the
// pass also returns the squared norm of the whole new residual.
micro_status execute_step(micro_ctx* ctx, const float* grad, float* residual, int64_t start, int64_t len,
                          bool accumulate_outside, double density, double* theta, int32_t* out_idx,
                          float* out_val, int64_t* k, double* sumsq) {
    DeviceScope scope(ctx->device);
    const micro_status checked = check_step_args(ctx, grad, residual, ctx->n_total, start, len, accumulate_outside,
                                                 density, theta, out_idx, out_val, k,
                                                 ctx->cfg.rule != MICRO_RULE_TOPK);
    if (checked != MICRO_OK) return checked;
    const int64_t n_outside = accumulate_outside ? ctx->n_total - len : 0;
    const bool topk = ctx->cfg.rule == MICRO_RULE_TOPK;
    if (len == 0 && n_outside == 0) {  // nothing to do: nothing selected, threshold unchanged
        *k = 0;
        if (sumsq) *sumsq = 0.0;
        return MICRO_OK;
    }
    if (sumsq) {
        // The pass with its local error: the whole vector through the sweep
        // kernels as three segments, the two outside the partition with a NaN
        // threshold (nothing selected, everything accumulated).
        if (!ctx->has_staged) {
            set_error(ctx, "the local error needs the staged schedule");
            return MICRO_EINVAL;
        }
        const float none = std::numeric_limits<float>::quiet_NaN();
        const int64_t starts[3] = {0, start, start + len};
        const int64_t lens[3] = {start, len, ctx->n_total - start - len};
        float thf[3] = {none, threshold_as_f32(*theta), none};
        TopkPlan plan;
        if (topk && len > 0) {
            if (ctx->needs_reset) {
                micro_status s = reset_scratch(ctx);
                if (s != MICRO_OK) return s;
            }
            const bool vec4 = ((reinterpret_cast<uintptr_t>(grad) ^ reinterpret_cast<uintptr_t>(residual)) & 15u) == 0;
            micro_status s = topk_plan(ctx, grad, residual, start, len, density, vec4, &plan);
            if (s != MICRO_OK) return s;
            thf[1] = plan.route == TopkRoute::kNone ? none : float_from_bits(plan.threshold_key);
        }
        int64_t kk[3];
        double sq[3];
        const micro_status st =
            run_segments(ctx, grad, residual, 3, starts, lens, thf, density * static_cast<double>(len), out_idx,
                         out_val, kk, sq);
        if (st != MICRO_OK) return st;
        if (kk[0] != 0 || kk[2] != 0) {
            set_error(ctx, "device selected outside the partition");
            ctx->needs_reset = true;
            return MICRO_EHIP;
        }
        if (topk) {
            if (plan.route == TopkRoute::kList || plan.trim) {
                hipError_t e = topk_after_step(ctx, plan, out_idx, out_val, residual);
                if (e != hipSuccess) return hip_fail(ctx, e, "top-k launch after the step");
                if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess)
                    return hip_fail(ctx, e, "hipStreamSynchronize");
            }
            double returned;
            const micro_status s = topk_finish(ctx, plan, kk[1], &kk[1], theta, &returned);
            if (s != MICRO_OK) return s;
            sq[1] += returned;  // the values the trim returned to the residual
            *k = kk[1];
            ctx->stats.topk_route = topk_route_code(plan.route);
        } else {
            *k = kk[1];
            *theta = next_threshold(ctx->cfg, density, len, kk[1], *theta);
        }
        *sumsq = sq[0] + sq[1] + sq[2];
        return MICRO_OK;
    }
    if (ctx->needs_reset) {
        micro_status s = reset_scratch(ctx);
        if (s != MICRO_OK) return s;
    }
    if (ctx->epoch >= micro::kMaxEpoch) {  // epoch field would wrap: clear the status words
        micro_status s = reset_scratch(ctx);
        if (s != MICRO_OK) return s;
    }
    const bool vec4 = ((reinterpret_cast<uintptr_t>(grad) ^ reinterpret_cast<uintptr_t>(residual)) & 15u) == 0;
    micro::AccumulateArgs acc{};
    if (n_outside > 0) {
        acc.grad = grad;
        acc.residual = residual;
        const int64_t lo[2] = {0, start + len}, hi[2] = {start, ctx->n_total};
        for (int r = 0; r < 2; ++r) {
            acc.start[r] = lo[r];
            acc.end[r] = hi[r];
            acc.base[r] = micro::tile_base_for(grad, lo[r], vec4);
            acc.tiles[r] = hi[r] > lo[r] ? static_cast<uint32_t>((hi[r] - acc.base[r] + micro::kStreamTile - 1) /
                                                                  micro::kStreamTile)
                                         : 0u;
        }
    }
    // AUTO contexts take the one-pass ticket schedule for partitions of up to
    // kAutoTicketMax values, where one launch beats three, and the staged
    // schedule above, where the ticket schedule's per-tile round trips cost
    // bandwidth.
    const bool staged = ctx->has_staged && !(ctx->has_ticket && len <= kAutoTicketMax);
    const int64_t tile_elems = staged ? micro::kStreamTile : micro::kTicketTile;
    micro::LaunchArgs a{};
    a.grad = grad;
    a.residual = residual;
    a.out_idx = out_idx;
    a.out_val = out_val;
    a.start = start;
    a.end = start + len;
    a.base = micro::tile_base_for(grad, start, vec4);
    a.theta_f = threshold_as_f32(*theta);
    a.epoch = ctx->epoch + 1;
    const int64_t tiles = len > 0 ? (a.end - a.base + tile_elems - 1) / tile_elems : 0;
    const int64_t chunks = (tiles + micro::kChunkTiles - 1) / micro::kChunkTiles;
    const int64_t capacity = staged ? ctx->tile_capacity : ctx->ticket_capacity;
    if (tiles > capacity || (staged && chunks > ctx->chunk_capacity)) {
        set_error(ctx, "partition needs %lld tiles, scratch holds %lld", static_cast<long long>(tiles),
                  static_cast<long long>(capacity));
        return MICRO_ECAPACITY;
    }
    a.num_tiles = static_cast<uint32_t>(tiles);
    a.count_out = ctx->d_count;
    a.host_count = ctx->h_count_dev;
    a.tile_counts = ctx->d_tile_counts;
    a.tile_words = ctx->d_tile_words;
    a.tile_excl = ctx->d_tile_excl;
    a.flagged_list = ctx->d_flagged_list;
    a.split_tile = ctx->d_split_tile;
    a.move_span = move_span_for(ctx, tiles, density * static_cast<double>(len));
    // Sized for twice the expected count (the count of the first steps under
    // error feedback), and at least four workgroups per compute unit so that
    // a count far above it still spreads over the device.  Against a grid for
    // the largest count, BERT-large rank 3 (1024 instead of 2048 workgroups):
    // 71.2% against 71.0% of 8 TB/s (medians of four runs each, one box),
    // within the run-to-run spread of about 1%: no slower, and fewer idle
    // workgroups.
    const double expected_pairs = density * static_cast<double>(len);
    a.move_blocks = move_grid(tiles, static_cast<int64_t>(std::min(static_cast<double>(len), 2.0 * expected_pairs)),
                              a.move_span, std::min<int64_t>(4 * ctx->compute_units, micro::kMoveGrid));
    a.stage = ctx->d_stage;
    a.num_chunks = static_cast<uint32_t>(chunks);
    a.chunk_status = ctx->d_chunk_status;
    a.status = ctx->d_status;
    a.ticket = &ctx->d_tickets[0];

    hipError_t e;
    const bool timed = (ctx->cfg.flags & MICRO_FLAG_TIME_KERNEL) != 0;
    ctx->stats.kernel_ms = -1.0f;
    ctx->stats.redone_tiles = 0;
    if (timed && (e = hipEventRecord(ctx->ev[0], ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "hipEventRecord");
    // The top-k comparator: with a hint the step runs at the hint's bound;
    // else the exact k-th largest magnitude, or its first digit's bin, first
    // (waited for), then the step there (NaN: nothing selected).
    TopkPlan plan;
    if (topk && len > 0) {
        uint32_t hint_key;
        if (topk_hint_key(ctx, *theta, topk_count(density, len), len, &hint_key)) {
            plan.route = TopkRoute::kHint;
            plan.threshold_key = hint_key;
            plan.zero_key = hint_key;
            if (staged) {  // the staged kernels leave acc in the residual below theta_zero
                a.theta_zero = f32_at_or_below(*theta);
                std::memcpy(&plan.zero_key, &a.theta_zero, sizeof plan.zero_key);
            }
        } else {
            micro_status s = topk_plan(ctx, grad, residual, start, len, density, vec4, &plan);
            if (s != MICRO_OK) return s;
        }
        a.theta_f = plan.route == TopkRoute::kNone ? std::numeric_limits<float>::quiet_NaN()
                                                   : float_from_bits(plan.threshold_key);
    }
    volatile int64_t* host_count = ctx->h_count;  // stored by the last kernel of the step
    host_count[0] = len > 0 ? -1 : 0;
    host_count[1] = len > 0 ? -1 : 0;
    if (n_outside > 0 && (e = micro::launch_accumulate(acc, vec4, ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "accumulate kernel launch");
    // The staged schedule's stream and scan kernels run as one launch unless
    // the caller asked for the scan on its own.
    const bool fused = staged && (ctx->cfg.flags & MICRO_FLAG_SEPARATE_SCAN) == 0;
    if (len > 0) {
        ctx->epoch = a.epoch;
        e = !staged ? micro::launch_ticket(a, vec4, ctx->stream)
            : fused ? micro::launch_fused(a, vec4, ctx->stream)
                    : micro::launch_staged(a, vec4, ctx->stream);
        if (e != hipSuccess) return hip_fail(ctx, e, "sparsify kernel launch");
    }
    // The top-k comparator's work after the step: on the hint's route, what
    // the step's count calls for; else the list route's last passes over the
    // step's output list, and the trim to the top k.
    if (topk && plan.route == TopkRoute::kHint) {
        if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess) return hip_fail(ctx, e, "hipStreamSynchronize");
        const int64_t listed = host_count[0];
        if (listed < 0 || listed > len) {
            set_error(ctx, "device reported %lld listed of %lld", static_cast<long long>(listed),
                      static_cast<long long>(len));
            ctx->needs_reset = true;
            return MICRO_EHIP;
        }
        const micro_status s = topk_after_hint(ctx, &plan, listed, residual, start, len, density, out_idx, out_val);
        if (s != MICRO_OK) return s;
    } else if (topk && (e = topk_after_step(ctx, plan, out_idx, out_val, residual)) != hipSuccess) {
        return hip_fail(ctx, e, "top-k launch after the step");
    }
    if (timed && (e = hipEventRecord(ctx->ev[1], ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "hipEventRecord");
    if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess) return hip_fail(ctx, e, "hipStreamSynchronize");
    int64_t selected = host_count[0];
    if (selected < 0 || selected > len) {
        set_error(ctx, "device reported %lld selected of %lld", static_cast<long long>(selected),
                  static_cast<long long>(len));
        ctx->needs_reset = true;
        return MICRO_EHIP;
    }
    if (topk) {
        const micro_status s = topk_finish(ctx, plan, selected, &selected, theta, nullptr);
        if (s != MICRO_OK) return s;
    }
    if (timed && (e = hipEventElapsedTime(&ctx->stats.kernel_ms, ctx->ev[0], ctx->ev[1])) != hipSuccess)
        return hip_fail(ctx, e, "hipEventElapsedTime");
    ctx->stats.redone_tiles = staged ? host_count[1] : 0;
    ctx->stats.variant = staged ? MICRO_VARIANT_STAGED : MICRO_VARIANT_TICKET;
    ctx->stats.fused = len > 0 && fused ? 1 : 0;
    ctx->stats.topk_route = topk ? topk_route_code(plan.route) : 0;
    *k = selected;
    if (!topk) *theta = next_threshold(ctx->cfg, density, len, selected, *theta);
    return MICRO_OK;
}

// One launch of each staged kernel over `count` segments of one vector: the
// segment [starts[r], starts[r] + lens[r]) selects with threshold_f[r] (a NaN
// threshold selects nothing: an ordered compare with NaN is false), all of
// them accumulate; the pairs of all segments form one compaction in index
// order.  k[r] and sumsq[r] (squared norm of the segment's new residual)
// receive each segment's results.  Arguments are validated by the callers.
micro_status run_segments(micro_ctx* ctx, const float* grad, float* residual, int32_t count, const int64_t* starts,
                          const int64_t* lens, const float* threshold_f, double expected_pairs, int32_t* out_idx,
                          float* out_val, int64_t* k, double* sumsq) {
    if (ctx->needs_reset || ctx->epoch >= micro::kMaxEpoch) {
        micro_status st = reset_scratch(ctx);
        if (st != MICRO_OK) return st;
    }
    const bool vec4 = ((reinterpret_cast<uintptr_t>(grad) ^ reinterpret_cast<uintptr_t>(residual)) & 15u) == 0;
    micro::SweepTable table{};
    table.count = static_cast<uint32_t>(count);
    int64_t tiles = 0, chunks = 0;
    for (int32_t r = 0; r < count; ++r) {
        micro::SweepSegment& sg = table.seg[r];
        sg.start = starts[r];
        sg.end = starts[r] + lens[r];
        sg.base = micro::tile_base_for(grad, starts[r], vec4);
        sg.theta_f = threshold_f[r];
        sg.tile_first = static_cast<uint32_t>(tiles);
        sg.chunk_first = static_cast<uint32_t>(chunks);
        sg.wg_first = static_cast<uint32_t>(tiles + chunks);  // the fused launch: segment after segment
        const int64_t seg_tiles = lens[r] > 0 ? (sg.end - sg.base + micro::kStreamTile - 1) / micro::kStreamTile : 0;
        tiles += seg_tiles;
        chunks += (seg_tiles + micro::kChunkTiles - 1) / micro::kChunkTiles;
    }
    table.seg[count].tile_first = static_cast<uint32_t>(tiles);
    table.seg[count].chunk_first = static_cast<uint32_t>(chunks);
    table.seg[count].wg_first = static_cast<uint32_t>(tiles + chunks);
    if (tiles > ctx->tile_capacity || chunks > ctx->chunk_capacity) {
        set_error(ctx, "sweep needs %lld tiles, scratch holds %lld", static_cast<long long>(tiles),
                  static_cast<long long>(ctx->tile_capacity));
        return MICRO_ECAPACITY;
    }
    if (tiles == 0) {  // every segment empty
        for (int32_t r = 0; r < count; ++r) {
            k[r] = 0;
            sumsq[r] = 0.0;
        }
        return MICRO_OK;
    }
    micro::LaunchArgs a{};
    a.grad = grad;
    a.residual = residual;
    a.out_idx = out_idx;
    a.out_val = out_val;
    a.epoch = ctx->epoch + 1;
    a.num_tiles = static_cast<uint32_t>(tiles);
    a.count_out = ctx->d_count;
    a.host_count = ctx->h_count_dev;
    a.tile_counts = ctx->d_tile_counts;
    a.tile_words = ctx->d_tile_words;
    a.tile_excl = ctx->d_tile_excl;
    a.flagged_list = ctx->d_flagged_list;
    a.split_tile = ctx->d_split_tile;
    a.tile_sumsq = ctx->d_tile_sumsq;
    a.host_sumsq = ctx->h_sumsq_dev;
    int64_t total_len = 0;
    for (int32_t r = 0; r < count; ++r) total_len += lens[r];
    a.move_span = move_span_for(ctx, tiles, expected_pairs);
    // workgroup r of the move kernel reduces segment r's squared norm
    a.move_blocks = move_grid(tiles, total_len, a.move_span, count);
    a.stage = ctx->d_stage;
    a.num_chunks = static_cast<uint32_t>(chunks);
    a.chunk_status = ctx->d_chunk_status;

    hipError_t e;
    const bool timed = (ctx->cfg.flags & MICRO_FLAG_TIME_KERNEL) != 0;
    ctx->stats.kernel_ms = -1.0f;
    ctx->stats.redone_tiles = 0;
    volatile int64_t* host_count = ctx->h_count;
    volatile double* host_sumsq = ctx->h_sumsq;
    for (int i = 0; i < 2 + count; ++i) host_count[i] = -1;
    for (int64_t c = 0; c < chunks; ++c) host_sumsq[c] = -1.0;
    // The stream and scan passes run as one launch for sweeps of up to
    // kFusedSweepMaxChunks scan chunks, unless the caller asked for the scan
    // on its own.
    const bool fused = (ctx->cfg.flags & MICRO_FLAG_SEPARATE_SCAN) == 0 && chunks <= kFusedSweepMaxChunks;
    if (timed && (e = hipEventRecord(ctx->ev[0], ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "hipEventRecord");
    ctx->epoch = a.epoch;
    if ((e = micro::launch_sweep(a, table, vec4, fused, ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "sweep kernel launch");
    if (timed && (e = hipEventRecord(ctx->ev[1], ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "hipEventRecord");
    if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess) return hip_fail(ctx, e, "hipStreamSynchronize");
    int64_t sum = 0;
    bool ok = host_count[0] >= 0 && host_count[0] <= ctx->n_total;
    for (int32_t r = 0; ok && r < count; ++r) {
        const int64_t kr = host_count[2 + r];
        ok = kr >= 0 && kr <= lens[r];
        sum += kr;
    }
    for (int64_t c = 0; ok && c < chunks; ++c) ok = host_sumsq[c] != -1.0;  // a NaN residual gives a NaN norm
    if (!ok || sum != host_count[0]) {
        set_error(ctx, "device reported inconsistent sweep counts (total %lld)",
                  static_cast<long long>(host_count[0]));
        ctx->needs_reset = true;
        return MICRO_EHIP;
    }
    if (timed && (e = hipEventElapsedTime(&ctx->stats.kernel_ms, ctx->ev[0], ctx->ev[1])) != hipSuccess)
        return hip_fail(ctx, e, "hipEventElapsedTime");
    ctx->stats.redone_tiles = host_count[1];
    ctx->stats.variant = MICRO_VARIANT_STAGED;
    ctx->stats.fused = fused ? 1 : 0;
    ctx->stats.topk_route = 0;
    for (int32_t r = 0; r < count; ++r) {
        k[r] = host_count[2 + r];
        // the segment's chunks in increasing order
        double sq = 0.0;
        for (uint32_t c = table.seg[r].chunk_first; c < table.seg[r + 1].chunk_first; ++c) sq += host_sumsq[c];
        sumsq[r] = sq;
    }
    return MICRO_OK;
}

// Every partition of `world` searched once in one launch of each staged
// kernel; the pairs of all partitions form one compaction in index order.
micro_status execute_sweep(micro_ctx* ctx, const float* grad, float* residual, int32_t world, double density,
                           double* theta, int32_t* out_idx, float* out_val, int64_t* k, double* sumsq) {
    DeviceScope scope(ctx->device);
    if (!grad || !residual || !theta || !out_idx || !out_val || !k) {
        set_error(ctx, "NULL pointer argument");
        return MICRO_EINVAL;
    }
    if (world < 1 || world > micro::kMaxSweep) {
        set_error(ctx, "sweep world %d outside [1, %d]", world, micro::kMaxSweep);
        return MICRO_EINVAL;
    }
    if (!ctx->has_staged) {
        set_error(ctx, "the sweep needs the staged schedule");
        return MICRO_EINVAL;
    }
    if (ctx->cfg.rule == MICRO_RULE_TOPK) {
        set_error(ctx, "the top-k comparator runs through micro_sparsify_step and micro_ef_step, not the sweep");
        return MICRO_EINVAL;
    }
    if (!density_valid(density)) {
        set_error(ctx, "density %g outside (0, 1]", density);
        return MICRO_EINVAL;
    }
    for (int32_t r = 0; r < world; ++r)
        if (!theta_valid(theta[r])) {
            set_error(ctx, "threshold %g of partition %d is not finite and positive", theta[r], r);
            return MICRO_EINVAL;
        }
    if (misaligned4({grad, residual, out_idx, out_val})) {
        set_error(ctx, "buffers must be 4-byte aligned");
        return MICRO_EINVAL;
    }
    const size_t nb = static_cast<size_t>(ctx->n_total) * sizeof(float);
    const void* regions[4] = {grad, residual, out_idx, out_val};
    for (int i = 0; i < 4; ++i)
        for (int j = i + 1; j < 4; ++j)
            if (nb > 0 && ranges_overlap(regions[i], nb, regions[j], nb)) {
                set_error(ctx, "grad, residual and output ranges overlap");
                return MICRO_EINVAL;
            }
    if (ctx->n_total == 0) {
        for (int32_t r = 0; r < world; ++r) {
            k[r] = 0;
            if (sumsq) sumsq[r] = 0.0;
        }
        return MICRO_OK;
    }
    int64_t starts[micro::kMaxSweep], lens[micro::kMaxSweep];
    float theta_f[micro::kMaxSweep];
    for (int32_t r = 0; r < world; ++r) {
        (void)micro_partition(ctx->n_total, r, world, &starts[r], &lens[r]);
        theta_f[r] = threshold_as_f32(theta[r]);
    }
    double sq[micro::kMaxSweep];
    const micro_status st = run_segments(ctx, grad, residual, world, starts, lens, theta_f,
                                         density * static_cast<double>(ctx->n_total), out_idx, out_val, k, sq);
    if (st != MICRO_OK) return st;
    for (int32_t r = 0; r < world; ++r) {
        theta[r] = next_threshold(ctx->cfg, density, lens[r], k[r], theta[r]);
        if (sumsq) sumsq[r] = sq[r];
    }
    return MICRO_OK;
}

// Enqueues one union kernel on the context's stream.  With the timing flag
// the call waits for it and records its duration; otherwise it returns after
// the launch.
template <class Launch>
micro_status execute_union(micro_ctx* ctx, Launch launch) {
    DeviceScope scope(ctx->device);
    hipError_t e;
    const bool timed = (ctx->cfg.flags & MICRO_FLAG_TIME_KERNEL) != 0;
    ctx->stats.kernel_ms = -1.0f;
    ctx->stats.redone_tiles = 0;
    if (timed && (e = hipEventRecord(ctx->ev[0], ctx->stream)) != hipSuccess)
        return hip_fail(ctx, e, "hipEventRecord");
    if ((e = launch(ctx->stream)) != hipSuccess) return hip_fail(ctx, e, "union kernel launch");
    if (timed) {
        if ((e = hipEventRecord(ctx->ev[1], ctx->stream)) != hipSuccess) return hip_fail(ctx, e, "hipEventRecord");
        if ((e = hipEventSynchronize(ctx->ev[1])) != hipSuccess) return hip_fail(ctx, e, "hipEventSynchronize");
        if ((e = hipEventElapsedTime(&ctx->stats.kernel_ms, ctx->ev[0], ctx->ev[1])) != hipSuccess)
            return hip_fail(ctx, e, "hipEventElapsedTime");
    }
    return MICRO_OK;
}

// The allocation-free step's state on one device: the address of the
// device's static scratch, the epoch of its last launch (the look-back words
// carry it, so they are cleared only when it would wrap), and whether the
// scratch must be cleared before the next launch (after a failure).  Calls on
// one device hold its mutex from validation of the scratch to the count
// readback, so they never overlap on the scratch.
struct NoallocDevice {
    std::mutex mutex;
    uint64_t* words = nullptr;
    uint32_t epoch = 0;
    bool needs_reset = false;
};

constexpr int kMaxNoallocDevices = 64;
NoallocDevice g_noalloc[kMaxNoallocDevices];

micro_status noalloc_fail(NoallocDevice& dv, hipError_t err, const char* what) {
    dv.needs_reset = true;
    return hip_fail(nullptr, err, what);
}

}  // namespace

extern "C" {

micro_status micro_sparsify_step_noalloc(const float* grad, float* residual, int64_t n_total, int32_t rank,
                                         int32_t world, double density, double* theta, int32_t* out_idx,
                                         float* out_val, int64_t* k, void* hip_stream, const micro_config* cfg) {
    micro_config c;
    micro_config_default(&c);
    if (cfg) c = *cfg;
    if (n_total < 0 || !config_valid(c)) {
        set_error(nullptr, "invalid n_total or configuration");
        return MICRO_EINVAL;
    }
    if (c.rule == MICRO_RULE_TOPK) {
        set_error(nullptr, "the top-k comparator needs a context (micro_sparsify_step)");
        return MICRO_EINVAL;
    }
    if (n_total > std::numeric_limits<int32_t>::max()) {
        set_error(nullptr, "n_total %lld exceeds 2^31 - 1 values, the int32 index range the static scratch covers",
                  static_cast<long long>(n_total));
        return MICRO_ERANGE;
    }
    int64_t start = 0, len = 0;
    if (micro_partition(n_total, rank, world, &start, &len) != MICRO_OK) {
        set_error(nullptr, "invalid rank %d / world %d", rank, world);
        return MICRO_EINVAL;
    }
    const micro_status checked =
        check_step_args(nullptr, grad, residual, n_total, start, len, false, density, theta, out_idx, out_val, k);
    if (checked != MICRO_OK) return checked;
    if (len == 0) {
        *k = 0;
        return MICRO_OK;
    }
    const bool vec4 = ((reinterpret_cast<uintptr_t>(grad) ^ reinterpret_cast<uintptr_t>(residual)) & 15u) == 0;
    micro::LaunchArgs a{};
    a.grad = grad;
    a.residual = residual;
    a.out_idx = out_idx;
    a.out_val = out_val;
    a.start = start;
    a.end = start + len;
    a.base = micro::tile_base_for(grad, start, vec4);
    a.theta_f = threshold_as_f32(*theta);
    const int64_t tiles = (a.end - a.base + micro::kTicketTile - 1) / micro::kTicketTile;
    if (tiles > micro::kStaticMaxTiles) {  // not reachable below 2^31 values; kept as the guard of the scratch
        set_error(nullptr, "partition needs %lld tiles, the static scratch holds %lld", static_cast<long long>(tiles),
                  static_cast<long long>(micro::kStaticMaxTiles));
        return MICRO_ECAPACITY;
    }
    a.num_tiles = static_cast<uint32_t>(tiles);
    int device = -1;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_fail(nullptr, e, "hipGetDevice");
    if (device < 0 || device >= kMaxNoallocDevices) {
        set_error(nullptr, "device %d is beyond the %d devices the static scratch tracks", device,
                  kMaxNoallocDevices);
        return MICRO_EHIP;
    }
    NoallocDevice& dv = g_noalloc[device];
    std::lock_guard<std::mutex> lock(dv.mutex);
    if (!dv.words && (e = micro::static_scratch_current_device(&dv.words)) != hipSuccess)
        return hip_fail(nullptr, e, "static scratch lookup (hipGetSymbolAddress)");
    const hipStream_t stream = static_cast<hipStream_t>(hip_stream);
    if (dv.needs_reset || dv.epoch >= micro::kMaxEpoch) {
        if ((e = micro::launch_clear_words(dv.words, micro::kStaticScratchWords, stream)) != hipSuccess)
            return noalloc_fail(dv, e, "static scratch clear");
        dv.epoch = 0;
    }
    a.ticket = reinterpret_cast<unsigned long long*>(dv.words);
    a.count_out = reinterpret_cast<int64_t*>(dv.words + 1);
    a.host_count = reinterpret_cast<int64_t*>(dv.words + 3);
    a.status = dv.words + micro::kStaticHeaderWords;
    a.epoch = dv.epoch + 1;
    if ((e = micro::launch_ticket(a, vec4, stream)) != hipSuccess) return noalloc_fail(dv, e, "sparsify kernel launch");
    dv.epoch = a.epoch;
    int64_t selected = -1;
    if ((e = hipMemcpyAsync(&selected, dv.words + 1, sizeof selected, hipMemcpyDeviceToHost, stream)) != hipSuccess)
        return noalloc_fail(dv, e, "count readback");
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return noalloc_fail(dv, e, "hipStreamSynchronize");
    if (selected < 0 || selected > len) {
        set_error(nullptr, "device reported %lld selected of %lld", static_cast<long long>(selected),
                  static_cast<long long>(len));
        dv.needs_reset = true;
        return MICRO_EHIP;
    }
    dv.needs_reset = false;
    *k = selected;
    *theta = next_threshold(c, density, len, selected, *theta);
    return MICRO_OK;
}

void micro_config_default(micro_config* cfg) {
    if (!cfg) return;
    cfg->rule = MICRO_RULE_PROPORTIONAL;
    cfg->beta = 0.1;
    cfg->lo = 0.5;
    cfg->hi = 2.0;
    cfg->alpha = 0.05;
    cfg->variant = MICRO_VARIANT_AUTO;
    cfg->flags = 0;
}

micro_status micro_partition(int64_t n_total, int32_t rank, int32_t world, int64_t* start,
                             int64_t* len) {
    if (!start || !len || world < 1 || rank < 0 || rank >= world || n_total < 0)
        return MICRO_EINVAL;
    // Sec. 4.1: equal contiguous ranges; the floor split keeps lengths within
    // one of each other when world does not divide n_total.  rank * n_total
    // stays below 2^62 for n_total < 2^31.
    const int64_t s = (static_cast<int64_t>(rank) * n_total) / world;
    const int64_t e = (static_cast<int64_t>(rank + 1) * n_total) / world;
    *start = s;
    *len = e - s;
    return MICRO_OK;
}

micro_status micro_estimate_threshold(const micro_config* cfg, double density, int64_t part_len,
                                      int64_t k, double* theta) {
    micro_config c;
    micro_config_default(&c);
    if (cfg) c = *cfg;
    if (!theta || !config_valid(c) || !density_valid(density) || part_len < 0 || k < 0 ||
        k > part_len || c.rule == MICRO_RULE_TOPK)  // the top-k threshold comes from the values
        return MICRO_EINVAL;
    *theta = next_threshold(c, density, part_len, k, *theta);
    return MICRO_OK;
}

micro_status micro_threshold_f32(double theta, float* theta_f) {
    if (!theta_f || !theta_valid(theta)) return MICRO_EINVAL;
    *theta_f = threshold_as_f32(theta);
    return MICRO_OK;
}

micro_status micro_sparsify_init(micro_ctx** out, int64_t n_total, void* hip_stream,
                                 const micro_config* cfg) {
    if (!out) {
        set_error(nullptr, "ctx output pointer is NULL");
        return MICRO_EINVAL;
    }
    *out = nullptr;
    micro_config c;
    micro_config_default(&c);
    if (cfg) c = *cfg;
    if (n_total < 0 || !config_valid(c)) {
        set_error(nullptr, "invalid n_total or configuration");
        return MICRO_EINVAL;
    }
    if (n_total > std::numeric_limits<int32_t>::max()) {
        set_error(nullptr, "n_total %lld exceeds the int32 index range",
                  static_cast<long long>(n_total));
        return MICRO_ERANGE;
    }
    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e != hipSuccess || count < 1) {
        set_error(nullptr, "no HIP device available (%s)",
                  e == hipSuccess ? "device count is 0" : hipGetErrorString(e));
        return MICRO_EHIP;
    }
    micro_ctx* ctx = new (std::nothrow) micro_ctx;
    if (!ctx) {
        set_error(nullptr, "out of host memory");
        return MICRO_ENOMEM;
    }
    ctx->n_total = n_total;
    ctx->stream = static_cast<hipStream_t>(hip_stream);
    ctx->cfg = c;
    if ((e = hipGetDevice(&ctx->device)) != hipSuccess) {
        set_error(nullptr, "hipGetDevice failed: %s", hipGetErrorString(e));
        release(ctx);
        return MICRO_EHIP;
    }
    if ((e = hipDeviceGetAttribute(&ctx->compute_units, hipDeviceAttributeMultiprocessorCount, ctx->device)) !=
            hipSuccess ||
        ctx->compute_units < 1) {
        set_error(nullptr, "compute unit count unavailable: %s", hipGetErrorString(e));
        release(ctx);
        return MICRO_EHIP;
    }
    // Scratch sized for the largest possible partition (the whole vector),
    // plus one tile for the alignment of the first tile.
    ctx->has_staged = c.variant != MICRO_VARIANT_TICKET;
    ctx->has_ticket = c.variant != MICRO_VARIANT_STAGED;
    bool ok = hipMalloc(&ctx->d_tickets, sizeof(unsigned long long)) == hipSuccess &&
              hipMalloc(&ctx->d_count, 2 * sizeof(int64_t)) == hipSuccess &&
              hipHostMalloc(&ctx->h_count, (2 + micro::kMaxSweep) * sizeof(int64_t),
                            hipHostMallocMapped | hipHostMallocCoherent) == hipSuccess &&
              hipHostGetDevicePointer(reinterpret_cast<void**>(&ctx->h_count_dev), ctx->h_count, 0) == hipSuccess &&
              hipMalloc(&ctx->d_topk, sizeof(uint32_t) * (micro::kTopkBins + micro::kTopkStateWords)) == hipSuccess &&
              hipHostMalloc(&ctx->h_topk, micro::kTopkHostWords * sizeof(int64_t),
                            hipHostMallocMapped | hipHostMallocCoherent) == hipSuccess &&
              hipHostGetDevicePointer(reinterpret_cast<void**>(&ctx->h_topk_dev), ctx->h_topk, 0) == hipSuccess;
    if (ok && ctx->has_staged) {
        // a sweep's segments each add at most one tile (alignment) and one chunk
        ctx->tile_capacity = n_total / micro::kStreamTile + 2 + micro::kMaxSweep;
        ctx->chunk_capacity = ctx->tile_capacity / micro::kChunkTiles + 2 + micro::kMaxSweep;
        // every piece, and one word past the largest move grid (each
        // workgroup reads its first piece's two words before it knows k)
        ctx->split_capacity = (ctx->tile_capacity + n_total) / micro::kMoveSpanTiny + 2;
        if (ctx->split_capacity < micro::kMoveGrid + 1) ctx->split_capacity = micro::kMoveGrid + 1;
        const size_t stage = static_cast<size_t>(ctx->tile_capacity) * micro::kStageCap;
        ok = hipMalloc(&ctx->d_tile_counts, sizeof(uint32_t) * ctx->tile_capacity) == hipSuccess &&
             hipMalloc(&ctx->d_tile_excl, sizeof(uint32_t) * ctx->tile_capacity) == hipSuccess &&
             hipMalloc(&ctx->d_flagged_list, sizeof(uint32_t) * ctx->tile_capacity) == hipSuccess &&
             hipMalloc(&ctx->d_split_tile, sizeof(uint32_t) * ctx->split_capacity) == hipSuccess &&
             hipMalloc(&ctx->d_tile_sumsq, sizeof(double) * ctx->tile_capacity) == hipSuccess &&
             hipHostMalloc(&ctx->h_sumsq, sizeof(double) * ctx->chunk_capacity,
                           hipHostMallocMapped | hipHostMallocCoherent) == hipSuccess &&
             hipHostGetDevicePointer(reinterpret_cast<void**>(&ctx->h_sumsq_dev), ctx->h_sumsq, 0) == hipSuccess &&
             hipMalloc(&ctx->d_stage, sizeof(uint2) * stage) == hipSuccess &&
             hipMalloc(&ctx->d_chunk_status, sizeof(uint64_t) * ctx->chunk_capacity) == hipSuccess &&
             hipMalloc(&ctx->d_tile_words, sizeof(uint64_t) * ctx->tile_capacity) == hipSuccess;
    }
    if (ok && ctx->has_ticket) {
        ctx->ticket_capacity = n_total / micro::kTicketTile + 2;
        ok = hipMalloc(&ctx->d_status, sizeof(uint64_t) * ctx->ticket_capacity) == hipSuccess;
    }
    if (!ok) {
        set_error(nullptr, "device or pinned host allocation failed");
        release(ctx);
        return MICRO_ENOMEM;
    }
    if (c.flags & MICRO_FLAG_TIME_KERNEL) {
        for (hipEvent_t& ev : ctx->ev) {
            if ((e = hipEventCreate(&ev)) != hipSuccess) {
                set_error(nullptr, "hipEventCreate failed: %s", hipGetErrorString(e));
                release(ctx);
                return MICRO_EHIP;
            }
        }
    }
    ctx->stats.kernel_ms = -1.0f;
    ctx->stats.redone_tiles = 0;
    ctx->stats.variant = ctx->has_staged ? MICRO_VARIANT_STAGED : MICRO_VARIANT_TICKET;
    ctx->stats.fused = 0;
    ctx->stats.topk_route = 0;
    if (reset_scratch(ctx) != MICRO_OK) {
        set_error(nullptr, "%s", ctx->last_error.c_str());
        release(ctx);
        return MICRO_EHIP;
    }
    *out = ctx;
    return MICRO_OK;
}

micro_status micro_sparsify_step(micro_ctx* ctx, const float* grad, float* residual, int32_t rank,
                                 int32_t world, double density, double* theta, int32_t* out_idx,
                                 float* out_val, int64_t* k) {
    if (!ctx) {
        set_error(nullptr, "ctx is NULL");
        return MICRO_EINVAL;
    }
    int64_t start = 0, len = 0;
    if (micro_partition(ctx->n_total, rank, world, &start, &len) != MICRO_OK) {
        set_error(ctx, "invalid rank %d / world %d", rank, world);
        return MICRO_EINVAL;
    }
    return execute_step(ctx, grad, residual, start, len, false, density, theta, out_idx, out_val, k, nullptr);
}

micro_status micro_sweep_step(micro_ctx* ctx, const float* grad, float* residual, int32_t world, double density,
                              double* theta, int32_t* out_idx, float* out_val, int64_t* k, double* sumsq) {
    if (!ctx) {
        set_error(nullptr, "ctx is NULL");
        return MICRO_EINVAL;
    }
    return execute_sweep(ctx, grad, residual, world, density, theta, out_idx, out_val, k, sumsq);
}

micro_status micro_cycle(int64_t t, int32_t worker, int32_t world, int32_t* cycle) {
    if (!cycle || t < 0 || world < 1 || worker < 0 || worker >= world) return MICRO_EINVAL;
    // Algorithm 1: the partition number advances by one every iteration.
    const int64_t n = world;
    *cycle = static_cast<int32_t>((t % n + worker) % n);
    return MICRO_OK;
}

micro_status micro_ef_step(micro_ctx* ctx, const float* grad, float* residual, int64_t t, int32_t worker,
                           int32_t world, double density, double* theta, int32_t* out_idx, float* out_val,
                           int64_t* k, int32_t* cycle, double* sumsq) {
    if (!ctx) {
        set_error(nullptr, "ctx is NULL");
        return MICRO_EINVAL;
    }
    int32_t part = 0;
    if (micro_cycle(t, worker, world, &part) != MICRO_OK) {
        set_error(ctx, "invalid iteration %lld / worker %d / world %d", static_cast<long long>(t), worker, world);
        return MICRO_EINVAL;
    }
    int64_t start = 0, len = 0;
    (void)micro_partition(ctx->n_total, part, world, &start, &len);
    const micro_status st =
        execute_step(ctx, grad, residual, start, len, true, density, theta, out_idx, out_val, k, sumsq);
    if (st == MICRO_OK && cycle) *cycle = part;
    return st;
}

micro_status micro_union_gather(micro_ctx* ctx, float* residual, const int32_t* union_idx, int64_t m,
                                int64_t own_first, int64_t own_count, const float* own_val, float* out) {
    if (!ctx) {
        set_error(nullptr, "ctx is NULL");
        return MICRO_EINVAL;
    }
    if (m < 0 || m > ctx->n_total || own_first < 0 || own_count < 0 || own_count > m - own_first) {
        set_error(ctx, "invalid union length %lld or own run [%lld, +%lld)", static_cast<long long>(m),
                  static_cast<long long>(own_first), static_cast<long long>(own_count));
        return MICRO_EINVAL;
    }
    if (m == 0) return MICRO_OK;
    if (!residual || !union_idx || !out || (own_count > 0 && !own_val)) {
        set_error(ctx, "NULL pointer argument");
        return MICRO_EINVAL;
    }
    if (misaligned4({residual, union_idx, own_val, out})) {
        set_error(ctx, "buffers must be 4-byte aligned");
        return MICRO_EINVAL;
    }
    const size_t mb = static_cast<size_t>(m) * 4, nb = static_cast<size_t>(ctx->n_total) * 4,
                 ob = static_cast<size_t>(own_count) * 4;
    if (ranges_overlap(out, mb, residual, nb) || ranges_overlap(out, mb, union_idx, mb) ||
        (own_count > 0 && (ranges_overlap(out, mb, own_val, ob) || ranges_overlap(residual, nb, own_val, ob))) ||
        ranges_overlap(residual, nb, union_idx, mb)) {
        set_error(ctx, "residual, union, own values and output overlap");
        return MICRO_EINVAL;
    }
    return execute_union(ctx, [&](hipStream_t s) {
        return micro::launch_union_gather(residual, ctx->n_total, union_idx, m, own_first, own_count, own_val,
                                          out, s);
    });
}

micro_status micro_sparse_update(micro_ctx* ctx, float* x, const int32_t* union_idx, const float* sums,
                                 int64_t m, int32_t world) {
    if (!ctx) {
        set_error(nullptr, "ctx is NULL");
        return MICRO_EINVAL;
    }
    if (m < 0 || m > ctx->n_total || world < 1) {
        set_error(ctx, "invalid union length %lld or world %d", static_cast<long long>(m), world);
        return MICRO_EINVAL;
    }
    if (m == 0) return MICRO_OK;
    if (!x || !union_idx || !sums) {
        set_error(ctx, "NULL pointer argument");
        return MICRO_EINVAL;
    }
    if (misaligned4({x, union_idx, sums})) {
        set_error(ctx, "buffers must be 4-byte aligned");
        return MICRO_EINVAL;
    }
    const size_t mb = static_cast<size_t>(m) * 4, nb = static_cast<size_t>(ctx->n_total) * 4;
    if (ranges_overlap(x, nb, union_idx, mb) || ranges_overlap(x, nb, sums, mb)) {
        set_error(ctx, "model, union and sums overlap");
        return MICRO_EINVAL;
    }
    const float n = static_cast<float>(world);
    return execute_union(ctx, [&](hipStream_t s) {
        return micro::launch_sparse_update(x, ctx->n_total, union_idx, sums, m, n, s);
    });
}

micro_status micro_sparsify_last_stats(const micro_ctx* ctx, micro_step_stats* stats) {
    if (!ctx || !stats) return MICRO_EINVAL;
    *stats = ctx->stats;
    return MICRO_OK;
}

const char* micro_last_error(const micro_ctx* ctx) {
    return ctx ? ctx->last_error.c_str() : g_init_error.c_str();
}

const char* micro_status_string(micro_status s) {
    switch (s) {
        case MICRO_OK: return "MICRO_OK";
        case MICRO_EINVAL: return "MICRO_EINVAL";
        case MICRO_ECAPACITY: return "MICRO_ECAPACITY";
        case MICRO_ERANGE: return "MICRO_ERANGE";
        case MICRO_ENOMEM: return "MICRO_ENOMEM";
        case MICRO_EHIP: return "MICRO_EHIP";
    }
    return "MICRO_UNKNOWN";
}

void micro_sparsify_free(micro_ctx* ctx) { release(ctx); }

}  // extern "C"
