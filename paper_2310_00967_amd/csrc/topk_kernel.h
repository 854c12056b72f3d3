// Internal interface of the exact top-k comparator's kernels (topk_kernel.hip).
// Not part of the C ABI.
//
// The comparator keeps the k accumulated values of largest magnitude of a
// partition (equal magnitudes: lower index first; NaN never).  Its k-th
// largest magnitude is found exactly by a radix select over the 31 magnitude
// bits of binary32 (for values that are not NaN, the bit pattern with the sign
// cleared orders like the magnitude), digits of 11, 11 and 9 bits, each digit
// by a histogram pass and a one-workgroup select.  The passes read their keys
// from acc = grad + residual over the partition, from the residual alone
// (once it holds acc), or from the values of the threshold step's output
// list, which holds every value at or above the step's threshold.  A trim
// then drops from that list the values below the k-th magnitude and the
// surplus of values equal to it; a pick instead takes the top k (or an
// extract every value from a bound up) straight from a residual that holds
// acc.
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
constexpr uint32_t kTopkFirstShift = 20;       // the first digit: key bits 30..20

// Device state words (after the kTopkBins counters):
enum TopkState : int {
    kTopkPrefix = 0,     // key bits fixed so far (the k-th key after the last pass)
    kTopkMask = 1,       // which key bits are fixed
    kTopkRemaining = 2,  // rank of the wanted key among the keys matching the prefix (1-based);
                         // after the last pass, the values equal to the k-th key that are kept
    kTopkValid = 3,      // values of the range that are not NaN
    kTopkGreater = 4,    // keys above the prefix's digit range so far: above the k-th key at the end
    kTopkEqual = 5,      // keys equal to the k-th key (after the last pass)
    kTopkStatus = 6,     // 0 searching, 1 found, 2 nothing to select
};

// Host words (mapped pinned memory), written by the select after the first
// pass with status 3 and after the last pass with status 1 (status 2:
// nothing to select): [0] the prefix (after the first pass: the first digit's
// bin, shifted in place; at the end the k-th key), [1] greater, [2] the
// count at the prefix (the first digit's bin, or the values equal to the
// k-th key), [3] remaining (at the end: the equal values kept), [4] valid,
// [5] status.  The trim writes [6], the bit pattern of the binary64 sum of
// squares of the values it returns to the residual.
struct TopkArgs {
    const float* grad;             // kAcc only
    const float* residual;
    int64_t start, end;            // the partition
    int64_t body_first, body_end;  // vec4: [body_first, body_end) in whole 16-byte groups of the vectors read
    bool vec4;
    uint32_t k;                    // the wanted count, 1 <= k <= the keys read
    const float* list;             // kList: the step's output values
    int64_t list_n;                // and their count
    uint32_t* words;               // kTopkBins counters (zero between passes), then kTopkStateWords
    int64_t* host;                 // kTopkHostWords mapped host words (device address)
    uint32_t blocks;               // grid of the histogram passes
};

// Where the histogram passes read their keys.
enum class TopkSource : int {
    kAcc = 0,       // acc = grad + residual over [start, end) (binary32 addition, as in the step)
    kResidual = 1,  // the residual alone over [start, end): it holds acc already
    kList = 2,      // list[0, list_n)
};

// Passes first .. last (0, 1, 2) of the radix select, each with its select.
// Pass 0 starts a new search: it reads no state of an earlier one.
hipError_t launch_topk_passes(const TopkArgs& args, TopkSource src, uint32_t first, uint32_t last,
                              hipStream_t stream);

// Drops from the index-ordered output list [0, n) the values whose key is
// below the k-th key, and those equal to it after the first `kept equal` of
// them (both read from the state words, after the last select), compacting
// the list, of which `kept` entries stay.  The step set the residual of the
// listed values with a key at or above zero_key to +0 and left acc in the
// others: a dropped value of the former returns to the residual, a kept value
// of the latter gets +0 there.  host[6] receives the binary64 sum of squares
// of the returned values.  With scratch (temp: n pairs; counts: two per kTopkTrimChunk list
// entries; partial: one per chunk) the whole device compacts the list in
// four launches: per chunk the equal and the lower keys counted, both counts
// scanned, every kept entry placed in temp and the dropped ones returned,
// temp copied back.  Without it (a null temp) one workgroup compacts the
// list in place, in order.
constexpr int kTopkTrimChunk = 4096;  // list entries per workgroup of the parallel trim
struct TopkTrimScratch {
    uint2* temp;       // >= n pairs
    uint32_t* counts;  // >= 2 * ceil(n / kTopkTrimChunk)
    double* partial;   // >= ceil(n / kTopkTrimChunk)
};
hipError_t launch_topk_trim(int32_t* out_idx, float* out_val, float* residual, int64_t n, int64_t kept,
                            uint32_t zero_key, const uint32_t* words, int64_t* host,
                            const TopkTrimScratch* scratch, hipStream_t stream);

// Writes the output list [0, n) back into the residual: residual[idx[j]] =
// val[j] for every idx[j] in [start, end) (the rest is skipped).  After the
// threshold step the residual then holds acc over the whole partition (the
// values the step did not set to +0 hold it already).
hipError_t launch_topk_restore(const int32_t* out_idx, const float* out_val, int64_t n, float* residual,
                               int64_t start, int64_t end, hipStream_t stream);

// Takes the top k straight from a residual holding acc over [start, end),
// after the last select: the values whose key is above the k-th key (NaN
// aside) and the first `kept equal` of those equal to it, in index order, into
// out_idx / out_val [0, kept), each replaced by +0 in the residual.  Three
// launches: per chunk of kTopkTrimChunk values the equal and the higher keys
// counted (counts: 2 * ceil((end - start) / kTopkTrimChunk) words), both
// counts scanned, every picked value placed.  Nothing is written without a
// k-th key (status other than 1).
hipError_t launch_topk_pick(float* residual, int64_t start, int64_t end, int32_t* out_idx, float* out_val,
                            const uint32_t* words, uint32_t* counts, hipStream_t stream);

// The same three launches with a fixed rule: every value of [start, end)
// whose key is at least key_floor (NaN aside) goes to out_idx / out_val in
// index order and its residual becomes +0 (the output holds at most
// end - start entries).
hipError_t launch_topk_extract(float* residual, int64_t start, int64_t end, uint32_t key_floor, int32_t* out_idx,
                               float* out_val, uint32_t* counts, hipStream_t stream);

}  // namespace micro
