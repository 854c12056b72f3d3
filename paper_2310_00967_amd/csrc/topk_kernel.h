// Internal interface of the exact top-k comparator's kernels (topk_kernel.hip).
// Not part of the C ABI.
//
// The comparator keeps the k accumulated values of largest magnitude of a
// partition (equal magnitudes: lower index first; NaN never).  Its k-th
// largest magnitude is found exactly by a radix select over the 31 magnitude
// bits of binary32 (for values that are not NaN, the bit pattern with the sign
// cleared orders like the magnitude): three histogram passes over
// acc = grad + residual, of 11, 11 and 9 bits, each followed by a
// one-workgroup select that fixes the digit holding the k-th key.  The
// selection itself is then the threshold step at that magnitude, and a trim
// pass drops the surplus of equal magnitudes from its output list.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace micro {

constexpr int kTopkBins = 2048;      // histogram counters (the widest digit, 11 bits)
constexpr int kTopkStateWords = 8;   // after the counters, in the same buffer
constexpr int kTopkHostWords = 8;    // the result as seen by the host
constexpr int kTopkHistBlock = 256;
constexpr int kTopkSelectBlock = 256;
constexpr int kTopkTrimBlock = 1024;
constexpr uint32_t kTopkKeyMax = 0x7F800000u;  // +inf with the sign cleared: larger keys are NaN

// Device state words (after the kTopkBins counters):
enum TopkState : int {
    kTopkPrefix = 0,     // key bits fixed so far
    kTopkMask = 1,       // which key bits are fixed
    kTopkRemaining = 2,  // rank of the wanted key among the keys matching the prefix (1-based)
    kTopkValid = 3,      // values of the range that are not NaN
    kTopkGreater = 4,    // keys above the prefix's digit range so far: above the k-th key at the end
    kTopkEqual = 5,      // keys equal to the k-th key (after the last pass)
    kTopkStatus = 6,     // 0 searching, 1 found, 2 nothing to select
};

// Host words (mapped pinned memory) written by the last select:
// [0] the k-th key, [1] greater, [2] equal, [3] m = the equal keys to keep,
// [4] valid, [5] status (1 found, 2 nothing).  The trim kernel writes
// [6] the bit pattern of the binary64 sum of squares of the values it
// returns to the residual.
struct TopkArgs {
    const float* grad;
    const float* residual;
    int64_t start, end;          // the partition
    int64_t body_first, body_end;  // vec4: [body_first, body_end) in whole 16-byte groups of both vectors
    bool vec4;
    uint32_t k;                  // the wanted count, 1 <= k <= end - start
    uint32_t* words;             // kTopkBins counters (zero between passes), then kTopkStateWords
    int64_t* host;               // kTopkHostWords mapped host words (device address)
    uint32_t blocks;             // grid of the histogram passes
};

// The three passes and selects (pass 0, 1, 2), enqueued on `stream`.
hipError_t launch_topk_select(const TopkArgs& args, hipStream_t stream);

// Drops from the index-ordered output list [0, n) the equal keys `key` after
// the first m of them, returning their values to the residual and compacting
// the list; host[6] receives the binary64 sum of squares of the returned
// values.  With scratch (temp: n pairs, counts and partial: one entry per
// kTopkTrimChunk list entries) the list is compacted by the whole device in
// four launches: ties counted per chunk, the counts scanned, every kept entry
// placed in temp and the dropped ones returned, temp copied back.  Without
// it (a null temp) one workgroup compacts the list in place, in order.
constexpr int kTopkTrimChunk = 4096;  // list entries per workgroup of the parallel trim
struct TopkTrimScratch {
    uint2* temp;       // >= n pairs
    uint32_t* counts;  // >= ceil(n / kTopkTrimChunk)
    double* partial;   // >= ceil(n / kTopkTrimChunk)
};
// kept: the entries that stay (n less the key-`key` entries after the first m).
hipError_t launch_topk_trim(int32_t* out_idx, float* out_val, float* residual, int64_t n, int64_t kept, uint32_t key,
                            int64_t m, int64_t* host, const TopkTrimScratch* scratch, hipStream_t stream);

}  // namespace micro
