// gfx950 kernels of the exact top-k comparator (the sorting-based sparsifier
// of Sec. 1 that keeps the k largest accumulated gradients; Sec. 2's error
// feedback supplies the values): a radix select of the k-th largest
// magnitude, the trim of the threshold step's output list, and the pick of
// the top k straight from the residual.  See topk_kernel.h.
#include "topk_kernel.h"

#include <type_traits>

namespace micro {
namespace {

using f32x4 = float __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// Where a histogram pass reads its keys.
constexpr int kSrcVec4 = 0;       // acc = grad + residual, 16-byte groups
constexpr int kSrcScalar = 1;     // acc = grad + residual, one value per load
constexpr int kSrcList = 2;       // the values of the step's output list
constexpr int kSrcResVec4 = 3;    // the residual alone (it holds acc), 16-byte groups
constexpr int kSrcResScalar = 4;  // the residual alone, one value per load

__device__ __forceinline__ uint32_t key_of(float v) {
    return __float_as_uint(v) & 0x7FFFFFFFu;
}

// Inclusive sum over the workgroup of one value per thread, in thread order;
// *total receives the workgroup's sum.  Contains two barriers.
template <int BLOCK>
__device__ __forceinline__ uint32_t block_inclusive_sum(uint32_t v, uint32_t* s_wave, uint32_t* total) {
    constexpr int WAVES = BLOCK / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const uint32_t o = __shfl_up(v, off, kWave);
        if (lane >= off) v += o;
    }
    if (lane == kWave - 1) s_wave[wave] = v;
    __syncthreads();
    uint32_t before = 0, sum = 0;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
        const uint32_t t = s_wave[w];
        if (w < wave) before += t;
        sum += t;
    }
    *total = sum;
    __syncthreads();  // s_wave is free again
    return before + v;
}

// Sum of one binary64 per thread over the workgroup in a fixed order (a
// butterfly in each wavefront, then the wavefronts in order); valid in
// thread 0.  Contains one barrier.
template <int WAVES>
__device__ __forceinline__ double block_sum_f64(double v, double* s_part) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    if ((threadIdx.x & (kWave - 1)) == 0) s_part[threadIdx.x / kWave] = v;
    __syncthreads();
    double total = 0.0;
    if (threadIdx.x == 0)
        for (int w = 0; w < WAVES; ++w) total += s_part[w];
    return total;
}

// Pass `pass` of the radix select: a histogram of one digit (bits 30..20,
// 19..9 or 8..0) of the keys that match the digits fixed by the earlier
// passes; NaN keys are not counted.  The keys are those of
// acc = grad + residual over [start, end) (binary32 addition, as in the
// step), of the residual alone there, or of the output list's values.  Each
// workgroup counts in LDS, then adds its nonzero counters to the global ones.
template <int SRC>
__global__ __launch_bounds__(kTopkHistBlock) void topk_hist_kernel(TopkArgs a, uint32_t pass) {
    constexpr bool kGrad = SRC == kSrcVec4 || SRC == kSrcScalar;
    __shared__ uint32_t s_hist[kTopkBins];
    const uint32_t* state = a.words + kTopkBins;
    uint32_t prefix = 0, mask = 0;
    if (pass > 0) {
        if (state[kTopkStatus] != 0) return;  // uniform: nothing left to find
        prefix = state[kTopkPrefix];
        mask = state[kTopkMask];
    }
    const uint32_t shift = pass == 0 ? kTopkFirstShift : pass == 1 ? 9u : 0u;
    const uint32_t digit = pass == 2 ? 511u : 2047u;
    for (int b = threadIdx.x; b < kTopkBins; b += kTopkHistBlock) s_hist[b] = 0u;
    __syncthreads();
    auto count_key = [&](uint32_t key) {
        if (key <= kTopkKeyMax && (key & mask) == prefix) atomicAdd(&s_hist[(key >> shift) & digit], 1u);
    };
    // acc at partition index i
    auto at = [&](int64_t i) {
        if constexpr (kGrad)
            return a.grad[i] + a.residual[i];
        else
            return a.residual[i];
    };
    const int64_t gtid = static_cast<int64_t>(blockIdx.x) * kTopkHistBlock + threadIdx.x;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kTopkHistBlock;
    if constexpr (SRC == kSrcVec4 || SRC == kSrcResVec4) {
        // the 16-byte groups of the body, two per thread in flight; fewer
        // than four values before and after it
        const f32x4* r4 = reinterpret_cast<const f32x4*>(a.residual + a.body_first);
        const f32x4* g4 = kGrad ? reinterpret_cast<const f32x4*>(a.grad + a.body_first) : r4;
        const int64_t groups = (a.body_end - a.body_first) / 4;
        int64_t q = gtid;
        for (; q + stride < groups; q += 2 * stride) {
            f32x4 v0, v1;
            if constexpr (kGrad) {
                const f32x4 g0 = __builtin_nontemporal_load(g4 + q);
                const f32x4 g1 = __builtin_nontemporal_load(g4 + q + stride);
                v0 = g0 + __builtin_nontemporal_load(r4 + q);
                v1 = g1 + __builtin_nontemporal_load(r4 + q + stride);
            } else {
                v0 = __builtin_nontemporal_load(r4 + q);
                v1 = __builtin_nontemporal_load(r4 + q + stride);
            }
#pragma unroll
            for (int c = 0; c < 4; ++c) count_key(key_of(v0[c]));
#pragma unroll
            for (int c = 0; c < 4; ++c) count_key(key_of(v1[c]));
        }
        if (q < groups) {
            f32x4 v0;
            if constexpr (kGrad)
                v0 = __builtin_nontemporal_load(g4 + q) + __builtin_nontemporal_load(r4 + q);
            else
                v0 = __builtin_nontemporal_load(r4 + q);
#pragma unroll
            for (int c = 0; c < 4; ++c) count_key(key_of(v0[c]));
        }
        if (gtid < a.body_first - a.start) count_key(key_of(at(a.start + gtid)));
        if (gtid < a.end - a.body_end) count_key(key_of(at(a.body_end + gtid)));
    } else if constexpr (SRC == kSrcScalar || SRC == kSrcResScalar) {
        for (int64_t i = a.start + gtid; i < a.end; i += stride) count_key(key_of(at(i)));
    } else {
        // the list's 16-byte groups, two per thread in flight (the list is
        // 4-byte aligned); fewer than four values before and after them
        const uintptr_t addr = reinterpret_cast<uintptr_t>(a.list);
        int64_t head = static_cast<int64_t>(((16u - (addr & 15u)) & 15u) / sizeof(float));
        if (head > a.list_n) head = a.list_n;
        const f32x4* l4 = reinterpret_cast<const f32x4*>(a.list + head);
        const int64_t groups = (a.list_n - head) / 4;
        int64_t q = gtid;
        for (; q + stride < groups; q += 2 * stride) {
            const f32x4 v0 = l4[q];
            const f32x4 v1 = l4[q + stride];
#pragma unroll
            for (int c = 0; c < 4; ++c) count_key(key_of(v0[c]));
#pragma unroll
            for (int c = 0; c < 4; ++c) count_key(key_of(v1[c]));
        }
        if (q < groups) {
            const f32x4 v0 = l4[q];
#pragma unroll
            for (int c = 0; c < 4; ++c) count_key(key_of(v0[c]));
        }
        const int64_t tail = head + groups * 4;
        if (gtid < head) count_key(key_of(a.list[gtid]));
        if (gtid < a.list_n - tail) count_key(key_of(a.list[tail + gtid]));
    }
    __syncthreads();
    for (int b = threadIdx.x; b < kTopkBins; b += kTopkHistBlock) {
        const uint32_t c = s_hist[b];
        if (c != 0u) atomicAdd(&a.words[b], c);
    }
}

// The select after pass `pass`, one workgroup: finds the digit value whose
// counter holds the wanted key (counting from the largest digit down), fixes
// it in the prefix and leaves the counters zero for the next pass.  Pass 0
// also counts the keys that are not NaN, caps the wanted rank by that count
// and reports its bin to the host; after pass 2 the prefix is the k-th key
// itself and the result goes to the host words.
__global__ __launch_bounds__(kTopkSelectBlock) void topk_select_kernel(TopkArgs a, uint32_t pass) {
    constexpr int PER = kTopkBins / kTopkSelectBlock;
    __shared__ uint32_t s_wave[kTopkSelectBlock / kWave];
    uint32_t* state = a.words + kTopkBins;
    const int tid = threadIdx.x;
    if (pass > 0 && state[kTopkStatus] != 0) return;  // uniform
    const uint32_t bins = pass == 2 ? 512u : static_cast<uint32_t>(kTopkBins);
    const uint32_t per = bins / kTopkSelectBlock;  // 8, or 2 for the last digit
    const uint32_t shift = pass == 0 ? kTopkFirstShift : pass == 1 ? 9u : 0u;
    const uint32_t digit = bins - 1;
    // thread t holds digits bins-1-t*per down to bins-(t+1)*per: thread order
    // is decreasing digit order
    uint32_t c[PER];
    uint32_t mine = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        c[i] = static_cast<uint32_t>(i) < per ? a.words[bins - 1 - (tid * per + i)] : 0u;
        mine += c[i];
    }
    uint32_t total;
    const uint32_t above_mine = block_inclusive_sum<kTopkSelectBlock>(mine, s_wave, &total) - mine;
    // every counter of this pass has been read (the sum's barriers): clear them
#pragma unroll
    for (int i = 0; i < PER; ++i)
        if (static_cast<uint32_t>(i) < per) a.words[bins - 1 - (tid * per + i)] = 0u;
    uint32_t remaining, prefix = 0, mask = 0, greater = 0;
    if (pass == 0) {
        remaining = total < a.k ? total : a.k;
        if (tid == 0) {
            state[kTopkValid] = total;
            state[kTopkStatus] = remaining == 0 ? 2u : 0u;
        }
        if (remaining == 0) {  // uniform: every value is NaN
            if (tid == 0) {
                a.host[4] = total;
                a.host[5] = 2;
            }
            return;
        }
    } else {
        remaining = state[kTopkRemaining];
        prefix = state[kTopkPrefix];
        mask = state[kTopkMask];
        greater = state[kTopkGreater];
    }
    if (above_mine < remaining && remaining <= above_mine + mine) {
        uint32_t above = above_mine;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            if (static_cast<uint32_t>(i) >= per) break;
            if (above + c[i] >= remaining) {
                const uint32_t d = bins - 1 - (tid * per + i);
                prefix |= d << shift;
                mask |= digit << shift;
                greater += above;
                remaining -= above;
                state[kTopkPrefix] = prefix;
                state[kTopkMask] = mask;
                state[kTopkGreater] = greater;
                state[kTopkRemaining] = remaining;
                if (pass == 2) {
                    state[kTopkEqual] = c[i];
                    state[kTopkStatus] = 1u;
                }
                if (pass == 0 || pass == 2) {
                    a.host[0] = prefix;
                    a.host[1] = greater;
                    a.host[2] = c[i];
                    a.host[3] = remaining;
                    a.host[4] = pass == 0 ? total : state[kTopkValid];
                    a.host[5] = pass == 0 ? 3 : 1;
                }
                break;
            }
            above += c[i];
        }
    }
}

// The trim's rule for an entry of the output list, given the k-th key `key`
// and the number `keep` of entries equal to it that stay: an entry with a
// lower key leaves; an entry equal to it leaves if `keep` equal entries come
// before it; every other entry moves left by the entries that left before it.
// The step set the residual of the listed values with a key at or above
// `zkey` to +0 and left acc in the others: a leaving entry of the former
// returns its value to the residual, a staying entry of the latter sets its
// residual to +0.

// One workgroup walks the list in chunks of kTopkTrimBlock * 4 entries, in
// order.  A chunk's entries are all read before any of its stores (the
// scans' barriers), and no store reaches beyond its entry's own position, so
// the later chunks still find their entries in place.
__global__ __launch_bounds__(kTopkTrimBlock) void topk_trim_kernel(int32_t* out_idx, float* out_val, float* residual,
                                                                   int64_t n, uint32_t zkey, const uint32_t* words,
                                                                   int64_t* host) {
    constexpr int PER = 4;
    constexpr int64_t CHUNK = static_cast<int64_t>(kTopkTrimBlock) * PER;
    constexpr int WAVES = kTopkTrimBlock / kWave;
    __shared__ uint32_t s_wave[WAVES];
    __shared__ double s_sq[WAVES];
    const uint32_t* state = words + kTopkBins;
    if (state[kTopkStatus] != 1u) return;  // uniform: no k-th key
    const uint32_t key = state[kTopkPrefix];
    const int64_t keep = state[kTopkRemaining];
    const int tid = threadIdx.x;
    int64_t ties_seen = 0, below_seen = 0;
    double sq = 0.0;
    for (int64_t base = 0; base < n; base += CHUNK) {  // uniform
        int32_t idx[PER];
        float val[PER];
        bool tie[PER], below[PER];
        uint32_t mine_t = 0, mine_b = 0;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int64_t pos = base + tid * PER + i;
            const bool live = pos < n;
            idx[i] = live ? out_idx[pos] : 0;
            val[i] = live ? out_val[pos] : 0.0f;
            tie[i] = live && key_of(val[i]) == key;
            below[i] = live && key_of(val[i]) < key;
            mine_t += tie[i] ? 1u : 0u;
            mine_b += below[i] ? 1u : 0u;
        }
        uint32_t chunk_t, chunk_b;
        const uint32_t incl_t = block_inclusive_sum<kTopkTrimBlock>(mine_t, s_wave, &chunk_t);
        const uint32_t incl_b = block_inclusive_sum<kTopkTrimBlock>(mine_b, s_wave, &chunk_b);
        int64_t rank = ties_seen + (incl_t - mine_t);
        int64_t lower = below_seen + (incl_b - mine_b);
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int64_t pos = base + tid * PER + i;
            if (pos >= n) break;
            const int64_t before_t = rank, before_b = lower;
            if (tie[i]) ++rank;
            if (below[i]) ++lower;
            if (below[i] || (tie[i] && before_t >= keep)) {
                if (key_of(val[i]) >= zkey) {
                    residual[idx[i]] = val[i];
                    sq += static_cast<double>(val[i]) * static_cast<double>(val[i]);
                }
            } else {
                if (key_of(val[i]) < zkey) residual[idx[i]] = 0.0f;
                const int64_t shift = before_b + (before_t > keep ? before_t - keep : 0);
                if (shift > 0) {
                    out_idx[pos - shift] = idx[i];
                    out_val[pos - shift] = val[i];
                }
            }
        }
        ties_seen += chunk_t;
        below_seen += chunk_b;
    }
    const double total = block_sum_f64<WAVES>(sq, s_sq);
    if (tid == 0) host[6] = static_cast<int64_t>(__double_as_longlong(total));
}

constexpr int kTrimBlock = 256;
constexpr int kTrimPer = kTopkTrimChunk / kTrimBlock;  // entries per thread, row j at j * kTrimBlock + thread
constexpr int kTrimWaves = kTrimBlock / kWave;

// Rows [J0, J0 + J) of a chunk whose first entry is v[base], of the entries
// before v[end] (end > 0): row j's entry at base + j * kTrimBlock + thread,
// or `pad` past end.  Every load is issued before any value is used (the
// index is clamped inside the array and the value replaced afterwards), so
// the loads of a thread overlap instead of each waiting for the last.
template <int J0, int J, class T>
__device__ __forceinline__ void load_rows(const T* v, int64_t base, int64_t end, T pad, T (&out)[J]) {
    const int64_t first = base + J0 * kTrimBlock + threadIdx.x;
    if (base + kTopkTrimChunk <= end) {  // uniform: a whole chunk
#pragma unroll
        for (int j = 0; j < J; ++j) out[j] = v[first + j * kTrimBlock];
    } else {
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int64_t p = first + j * kTrimBlock;
            out[j] = v[p < end ? p : end - 1];
        }
#pragma unroll
        for (int j = 0; j < J; ++j)
            if (first + j * kTrimBlock >= end) out[j] = pad;
    }
}

// Parallel trim, launch 1: per chunk of kTopkTrimChunk list entries, the
// entries equal to the k-th key (counts[chunk]) and below it
// (counts[chunks + chunk]).
__global__ __launch_bounds__(kTrimBlock) void topk_trim_count_kernel(const float* out_val, int64_t n,
                                                                     const uint32_t* words, uint32_t* counts,
                                                                     uint32_t chunks) {
    __shared__ uint32_t s_wave[kTrimWaves];
    const uint32_t* state = words + kTopkBins;
    if (state[kTopkStatus] != 1u) return;  // uniform
    const uint32_t key = state[kTopkPrefix];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kTopkTrimChunk;
    float v[kTrimPer];
    load_rows<0>(out_val, base, n, __uint_as_float(0xFFFFFFFFu), v);  // padding: a NaN key, neither count
    uint32_t t = 0, b = 0;
#pragma unroll
    for (int j = 0; j < kTrimPer; ++j) {
        const uint32_t kv = key_of(v[j]);
        t += kv == key ? 1u : 0u;
        b += kv < key ? 1u : 0u;
    }
    uint32_t total_t, total_b;
    block_inclusive_sum<kTrimBlock>(t, s_wave, &total_t);
    block_inclusive_sum<kTrimBlock>(b, s_wave, &total_b);
    if (threadIdx.x == 0) {
        counts[blockIdx.x] = total_t;
        counts[chunks + blockIdx.x] = total_b;
    }
}

// Launch 2, one workgroup: both count arrays become exclusive prefix sums,
// kScanPer consecutive counts of each array a thread (all loaded before any
// is used), one workgroup scan per kTopkTrimBlock * kScanPer counts.
constexpr int kScanPer = 16;
__global__ __launch_bounds__(kTopkTrimBlock) void topk_trim_scan_kernel(uint32_t* counts, uint32_t chunks) {
    __shared__ uint32_t s_wave[kTopkTrimBlock / kWave];
    constexpr uint32_t SPAN = static_cast<uint32_t>(kTopkTrimBlock) * kScanPer;
    uint32_t* c0 = counts;
    uint32_t* c1 = counts + chunks;
    uint32_t carry0 = 0, carry1 = 0;
    for (uint32_t base = 0; base < chunks; base += SPAN) {  // uniform
        const uint32_t first = base + threadIdx.x * kScanPer;
        uint32_t v0[kScanPer], v1[kScanPer];
#pragma unroll
        for (int i = 0; i < kScanPer; ++i) {
            const uint32_t j = first + i;
            v0[i] = j < chunks ? c0[j] : 0u;
            v1[i] = j < chunks ? c1[j] : 0u;
        }
        uint32_t sum0 = 0, sum1 = 0;
#pragma unroll
        for (int i = 0; i < kScanPer; ++i) {
            sum0 += v0[i];
            sum1 += v1[i];
        }
        uint32_t total0, total1;
        uint32_t run0 = carry0 + block_inclusive_sum<kTopkTrimBlock>(sum0, s_wave, &total0) - sum0;
        uint32_t run1 = carry1 + block_inclusive_sum<kTopkTrimBlock>(sum1, s_wave, &total1) - sum1;
#pragma unroll
        for (int i = 0; i < kScanPer; ++i) {
            const uint32_t j = first + i;
            if (j < chunks) {
                c0[j] = run0;
                c1[j] = run1;
            }
            run0 += v0[i];
            run1 += v1[i];
        }
        carry0 += total0;
        carry1 += total1;
    }
}

// Launch 3: each entry's counts of equal and lower entries before it (its
// chunk's prefixes, then rows in order and lanes in order inside the chunk)
// decide it: a dropped entry returns to the residual (at or above zkey), a
// kept one goes to temp at its position less the entries dropped before it
// (and below zkey sets its residual to +0).  partial[chunk] receives the
// binary64 sum of squares of the returned values.
__global__ __launch_bounds__(kTrimBlock) void topk_trim_scatter_kernel(const int32_t* out_idx, const float* out_val,
                                                                       float* residual, int64_t n, uint32_t zkey,
                                                                       const uint32_t* words,
                                                                       const uint32_t* counts, uint32_t chunks,
                                                                       uint2* temp, double* partial) {
    constexpr int ROWS = kTrimPer * kTrimWaves;
    static_assert(ROWS == kWave, "one (row, wavefront) count per lane of wavefront 0");
    __shared__ uint32_t s_t[ROWS], s_b[ROWS];
    __shared__ double s_sq[kTrimWaves];
    const uint32_t* state = words + kTopkBins;
    if (state[kTopkStatus] != 1u) return;  // uniform
    const uint32_t key = state[kTopkPrefix];
    const int64_t keep = state[kTopkRemaining];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kTopkTrimChunk;
    const uint64_t lower_lanes = lane ? (~0ull >> (kWave - lane)) : 0ull;
    // the chunk's prefixes, read before they are needed
    const int64_t chunk_t = counts[blockIdx.x], chunk_b = counts[chunks + blockIdx.x];
    uint32_t rank_t[kTrimPer], rank_b[kTrimPer];
    bool tie[kTrimPer], below[kTrimPer];
    {
        float v[kTrimPer];
        load_rows<0>(out_val, base, n, __uint_as_float(0xFFFFFFFFu), v);
#pragma unroll
        for (int j = 0; j < kTrimPer; ++j) {
            const uint32_t kv = key_of(v[j]);
            tie[j] = kv == key;
            below[j] = kv < key;
        }
    }
#pragma unroll
    for (int j = 0; j < kTrimPer; ++j) {
        const uint64_t mt = __ballot(tie[j]);
        const uint64_t mb = __ballot(below[j]);
        rank_t[j] = static_cast<uint32_t>(__popcll(mt & lower_lanes));
        rank_b[j] = static_cast<uint32_t>(__popcll(mb & lower_lanes));
        if (lane == 0) {
            s_t[j * kTrimWaves + wave] = static_cast<uint32_t>(__popcll(mt));
            s_b[j * kTrimWaves + wave] = static_cast<uint32_t>(__popcll(mb));
        }
    }
    __syncthreads();
    if (wave == 0) {  // exclusive prefixes of the (row, wavefront) counts, in list order
        uint32_t vt = s_t[lane], vb = s_b[lane];
        const uint32_t own_t = vt, own_b = vb;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
            const uint32_t ot = __shfl_up(vt, off, kWave);
            const uint32_t ob = __shfl_up(vb, off, kWave);
            if (lane >= off) {
                vt += ot;
                vb += ob;
            }
        }
        s_t[lane] = vt - own_t;
        s_b[lane] = vb - own_b;
    }
    __syncthreads();
    double sq = 0.0;
    // two halves of the rows, each with its loads issued together
    auto place = [&](auto half) {
        constexpr int J0 = decltype(half)::value * (kTrimPer / 2);
        int32_t idx[kTrimPer / 2];
        float val[kTrimPer / 2];
        load_rows<J0>(out_idx, base, n, int32_t(0), idx);
        load_rows<J0>(out_val, base, n, 0.0f, val);
#pragma unroll
        for (int u = 0; u < kTrimPer / 2; ++u) {
            const int j = J0 + u;
            const int64_t p = base + j * kTrimBlock + threadIdx.x;
            if (p >= n) continue;
            const int64_t before_t = chunk_t + s_t[j * kTrimWaves + wave] + rank_t[j];
            const int64_t before_b = chunk_b + s_b[j * kTrimWaves + wave] + rank_b[j];
            if (below[j] || (tie[j] && before_t >= keep)) {
                if (key_of(val[u]) >= zkey) {
                    residual[idx[u]] = val[u];
                    sq += static_cast<double>(val[u]) * static_cast<double>(val[u]);
                }
            } else {
                if (key_of(val[u]) < zkey) residual[idx[u]] = 0.0f;
                const int64_t to = p - before_b - (before_t > keep ? before_t - keep : 0);
                temp[to] = make_uint2(static_cast<uint32_t>(idx[u]), __float_as_uint(val[u]));
            }
        }
    };
    place(std::integral_constant<int, 0>{});
    place(std::integral_constant<int, 1>{});
    const double total = block_sum_f64<kTrimWaves>(sq, s_sq);
    if (threadIdx.x == 0) partial[blockIdx.x] = total;
}

// Launch 4: temp[0, kept) back into the output lists; workgroup 0 also adds
// the chunks' partial sums in a fixed order into host[6].
__global__ __launch_bounds__(kTrimBlock) void topk_trim_copy_kernel(const uint2* temp, int64_t kept, int32_t* out_idx,
                                                                    float* out_val, const uint32_t* words,
                                                                    const double* partial, uint32_t chunks,
                                                                    int64_t* host) {
    __shared__ double s_sq[kTrimWaves];
    if (words[kTopkBins + kTopkStatus] != 1u) return;  // uniform
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kTrimBlock;
    for (int64_t p = static_cast<int64_t>(blockIdx.x) * kTrimBlock + threadIdx.x; p < kept; p += stride) {
        const uint2 e = temp[p];
        out_idx[p] = static_cast<int32_t>(e.x);
        out_val[p] = __uint_as_float(e.y);
    }
    if (blockIdx.x == 0) {  // uniform
        double sq = 0.0;
        for (uint32_t c = threadIdx.x; c < chunks; c += kTrimBlock) sq += partial[c];
        const double total = block_sum_f64<kTrimWaves>(sq, s_sq);
        if (threadIdx.x == 0) host[6] = static_cast<int64_t>(__double_as_longlong(total));
    }
}

// Writes the output list back into the residual (one entry a thread, grid
// stride); indices outside [start, end) are skipped.
__global__ __launch_bounds__(kTrimBlock) void topk_restore_kernel(const int32_t* out_idx, const float* out_val,
                                                                  int64_t n, float* residual, int64_t start,
                                                                  int64_t end) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kTrimBlock;
    for (int64_t p = static_cast<int64_t>(blockIdx.x) * kTrimBlock + threadIdx.x; p < n; p += stride) {
        const int64_t i = out_idx[p];
        if (i >= start && i < end) residual[i] = out_val[p];
    }
}

// What a pick takes: the values whose key is above `key`, and the first
// `keep` of those equal to it, NaN aside.  With `words` the key and keep are
// the last select's (nothing is taken without a k-th key); without, they are
// the fixed ones here.
struct PickRule {
    const uint32_t* words;
    uint32_t key;
    int64_t keep;
};

__device__ __forceinline__ bool pick_rule(const PickRule& r, uint32_t& key, int64_t& keep) {
    if (r.words) {
        const uint32_t* state = r.words + kTopkBins;
        if (state[kTopkStatus] != 1u) return false;
        key = state[kTopkPrefix];
        keep = state[kTopkRemaining];
    } else {
        key = r.key;
        keep = r.keep;
    }
    return true;
}

// The pick, launch 1: per chunk of kTopkTrimChunk values of [start, end) of
// the residual, the values equal to the k-th key (counts[chunk]) and above it,
// NaN aside (counts[chunks + chunk]).
__global__ __launch_bounds__(kTrimBlock) void topk_pick_count_kernel(const float* residual, int64_t start,
                                                                     int64_t end, PickRule rule,
                                                                     uint32_t* counts, uint32_t chunks) {
    __shared__ uint32_t s_wave[kTrimWaves];
    uint32_t key;
    int64_t keep;
    if (!pick_rule(rule, key, keep)) return;  // uniform
    const int64_t base = start + static_cast<int64_t>(blockIdx.x) * kTopkTrimChunk;
    float v[kTrimPer];
    load_rows<0>(residual, base, end, __uint_as_float(0xFFFFFFFFu), v);  // padding: a NaN key, neither count
    uint32_t t = 0, h = 0;
#pragma unroll
    for (int j = 0; j < kTrimPer; ++j) {
        const uint32_t kv = key_of(v[j]);
        t += kv == key ? 1u : 0u;
        h += kv > key && kv <= kTopkKeyMax ? 1u : 0u;
    }
    uint32_t total_t, total_h;
    block_inclusive_sum<kTrimBlock>(t, s_wave, &total_t);
    block_inclusive_sum<kTrimBlock>(h, s_wave, &total_h);
    if (threadIdx.x == 0) {
        counts[blockIdx.x] = total_t;
        counts[chunks + blockIdx.x] = total_h;
    }
}

// Launch 3 (launch 2 is the trim's scan): each value's counts of equal and
// higher values before it (its chunk's prefixes, then rows in order and lanes
// in order inside the chunk) decide it.  A value above the k-th key, or equal
// to it with fewer than `keep` equal ones before it, is picked: it goes to the
// output at the number of values picked before it, and its residual becomes
// +0.  The placement never reaches past end - start entries.
__global__ __launch_bounds__(kTrimBlock) void topk_pick_scatter_kernel(float* residual, int64_t start, int64_t end,
                                                                       PickRule rule,
                                                                       const uint32_t* counts, uint32_t chunks,
                                                                       int32_t* out_idx, float* out_val) {
    constexpr int ROWS = kTrimPer * kTrimWaves;
    static_assert(ROWS == kWave, "one (row, wavefront) count per lane of wavefront 0");
    __shared__ uint32_t s_t[ROWS], s_h[ROWS];
    uint32_t key;
    int64_t keep;
    if (!pick_rule(rule, key, keep)) return;  // uniform
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t base = start + static_cast<int64_t>(blockIdx.x) * kTopkTrimChunk;
    const uint64_t lower_lanes = lane ? (~0ull >> (kWave - lane)) : 0ull;
    const int64_t chunk_t = counts[blockIdx.x], chunk_h = counts[chunks + blockIdx.x];
    uint32_t rank_t[kTrimPer], rank_h[kTrimPer];
    bool tie[kTrimPer], high[kTrimPer];
    float val[kTrimPer];
    load_rows<0>(residual, base, end, __uint_as_float(0xFFFFFFFFu), val);  // padding: a NaN key
#pragma unroll
    for (int j = 0; j < kTrimPer; ++j) {
        const uint32_t kv = key_of(val[j]);
        tie[j] = kv == key;
        high[j] = kv > key && kv <= kTopkKeyMax;
    }
#pragma unroll
    for (int j = 0; j < kTrimPer; ++j) {
        const uint64_t mt = __ballot(tie[j]);
        const uint64_t mh = __ballot(high[j]);
        rank_t[j] = static_cast<uint32_t>(__popcll(mt & lower_lanes));
        rank_h[j] = static_cast<uint32_t>(__popcll(mh & lower_lanes));
        if (lane == 0) {
            s_t[j * kTrimWaves + wave] = static_cast<uint32_t>(__popcll(mt));
            s_h[j * kTrimWaves + wave] = static_cast<uint32_t>(__popcll(mh));
        }
    }
    __syncthreads();
    if (wave == 0) {  // exclusive prefixes of the (row, wavefront) counts, in index order
        uint32_t vt = s_t[lane], vh = s_h[lane];
        const uint32_t own_t = vt, own_h = vh;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
            const uint32_t ot = __shfl_up(vt, off, kWave);
            const uint32_t oh = __shfl_up(vh, off, kWave);
            if (lane >= off) {
                vt += ot;
                vh += oh;
            }
        }
        s_t[lane] = vt - own_t;
        s_h[lane] = vh - own_h;
    }
    __syncthreads();
    const int64_t cap = end - start;
#pragma unroll
    for (int j = 0; j < kTrimPer; ++j) {
        const int64_t p = base + j * kTrimBlock + threadIdx.x;
        if (p >= end) continue;
        const int64_t before_t = chunk_t + s_t[j * kTrimWaves + wave] + rank_t[j];
        const int64_t before_h = chunk_h + s_h[j * kTrimWaves + wave] + rank_h[j];
        if (high[j] || (tie[j] && before_t < keep)) {
            const int64_t to = before_h + (before_t < keep ? before_t : keep);
            if (to < cap) {
                out_idx[to] = static_cast<int32_t>(p);
                out_val[to] = val[j];
                residual[p] = 0.0f;
            }
        }
    }
}

bool range_args_ok(const TopkArgs& a, bool grad) {
    return (!grad || a.grad) && a.residual && a.words && a.host && a.blocks > 0 && a.end > a.start && a.k > 0 &&
           (!a.vec4 || (a.body_first >= a.start && a.body_end >= a.body_first && a.body_end <= a.end &&
                        (a.body_end - a.body_first) % 4 == 0 && a.body_first - a.start <= 3 &&
                        a.end - a.body_end <= 3));
}

void launch_pass(const TopkArgs& a, TopkSource src, uint32_t pass, hipStream_t stream) {
    const dim3 grid(a.blocks), block(kTopkHistBlock);
    switch (src) {
    case TopkSource::kAcc:
        if (a.vec4)
            hipLaunchKernelGGL(topk_hist_kernel<kSrcVec4>, grid, block, 0, stream, a, pass);
        else
            hipLaunchKernelGGL(topk_hist_kernel<kSrcScalar>, grid, block, 0, stream, a, pass);
        break;
    case TopkSource::kResidual:
        if (a.vec4)
            hipLaunchKernelGGL(topk_hist_kernel<kSrcResVec4>, grid, block, 0, stream, a, pass);
        else
            hipLaunchKernelGGL(topk_hist_kernel<kSrcResScalar>, grid, block, 0, stream, a, pass);
        break;
    case TopkSource::kList:
        hipLaunchKernelGGL(topk_hist_kernel<kSrcList>, grid, block, 0, stream, a, pass);
        break;
    }
    hipLaunchKernelGGL(topk_select_kernel, dim3(1), dim3(kTopkSelectBlock), 0, stream, a, pass);
}

}  // namespace

hipError_t launch_topk_passes(const TopkArgs& a, TopkSource src, uint32_t first, uint32_t last, hipStream_t stream) {
    if (first > last || last > 2) return hipErrorInvalidValue;
    const bool ok = src == TopkSource::kList ? a.list && a.list_n >= 1 && a.k > 0 && a.words && a.host && a.blocks > 0
                                             : range_args_ok(a, src == TopkSource::kAcc);
    if (!ok) return hipErrorInvalidValue;
    for (uint32_t pass = first; pass <= last; ++pass) launch_pass(a, src, pass, stream);
    return hipGetLastError();
}

hipError_t launch_topk_trim(int32_t* out_idx, float* out_val, float* residual, int64_t n, int64_t kept,
                            uint32_t zero_key, const uint32_t* words, int64_t* host,
                            const TopkTrimScratch* scratch, hipStream_t stream) {
    if (!out_idx || !out_val || !residual || !words || !host || n <= 0 || kept < 1 || kept > n)
        return hipErrorInvalidValue;
    if (!scratch || !scratch->temp) {
        hipLaunchKernelGGL(topk_trim_kernel, dim3(1), dim3(kTopkTrimBlock), 0, stream, out_idx, out_val, residual, n,
                           zero_key, words, host);
        return hipGetLastError();
    }
    if (!scratch->counts || !scratch->partial) return hipErrorInvalidValue;
    const int64_t chunks = (n + kTopkTrimChunk - 1) / kTopkTrimChunk;
    if (chunks > 0x7FFFFFFFll) return hipErrorInvalidValue;
    const uint32_t nc = static_cast<uint32_t>(chunks);
    hipLaunchKernelGGL(topk_trim_count_kernel, dim3(nc), dim3(kTrimBlock), 0, stream, out_val, n, words,
                       scratch->counts, nc);
    hipLaunchKernelGGL(topk_trim_scan_kernel, dim3(1), dim3(kTopkTrimBlock), 0, stream, scratch->counts, nc);
    hipLaunchKernelGGL(topk_trim_scatter_kernel, dim3(nc), dim3(kTrimBlock), 0, stream, out_idx, out_val, residual,
                       n, zero_key, words, scratch->counts, nc, scratch->temp, scratch->partial);
    const uint32_t copy_blocks = nc < 2048u ? nc : 2048u;
    hipLaunchKernelGGL(topk_trim_copy_kernel, dim3(copy_blocks), dim3(kTrimBlock), 0, stream, scratch->temp, kept,
                       out_idx, out_val, words, scratch->partial, nc, host);
    return hipGetLastError();
}

hipError_t launch_topk_restore(const int32_t* out_idx, const float* out_val, int64_t n, float* residual,
                               int64_t start, int64_t end, hipStream_t stream) {
    if (!out_idx || !out_val || !residual || n < 0 || start < 0 || end < start) return hipErrorInvalidValue;
    if (n == 0) return hipSuccess;
    const int64_t blocks = (n + kTrimBlock - 1) / kTrimBlock;
    hipLaunchKernelGGL(topk_restore_kernel, dim3(static_cast<uint32_t>(blocks < 2048 ? blocks : 2048)),
                       dim3(kTrimBlock), 0, stream, out_idx, out_val, n, residual, start, end);
    return hipGetLastError();
}

namespace {

hipError_t launch_pick(float* residual, int64_t start, int64_t end, int32_t* out_idx, float* out_val,
                       const PickRule& rule, uint32_t* counts, hipStream_t stream) {
    if (!residual || !out_idx || !out_val || !counts || start < 0 || end <= start) return hipErrorInvalidValue;
    const int64_t chunks = (end - start + kTopkTrimChunk - 1) / kTopkTrimChunk;
    if (chunks > 0x7FFFFFFFll) return hipErrorInvalidValue;
    const uint32_t nc = static_cast<uint32_t>(chunks);
    hipLaunchKernelGGL(topk_pick_count_kernel, dim3(nc), dim3(kTrimBlock), 0, stream, residual, start, end, rule,
                       counts, nc);
    hipLaunchKernelGGL(topk_trim_scan_kernel, dim3(1), dim3(kTopkTrimBlock), 0, stream, counts, nc);
    hipLaunchKernelGGL(topk_pick_scatter_kernel, dim3(nc), dim3(kTrimBlock), 0, stream, residual, start, end, rule,
                       counts, nc, out_idx, out_val);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_topk_pick(float* residual, int64_t start, int64_t end, int32_t* out_idx, float* out_val,
                            const uint32_t* words, uint32_t* counts, hipStream_t stream) {
    if (!words) return hipErrorInvalidValue;
    return launch_pick(residual, start, end, out_idx, out_val, PickRule{words, 0u, 0}, counts, stream);
}

hipError_t launch_topk_extract(float* residual, int64_t start, int64_t end, uint32_t key_floor, int32_t* out_idx,
                               float* out_val, uint32_t* counts, hipStream_t stream) {
    if (key_floor > kTopkKeyMax) return hipErrorInvalidValue;
    // every key above the floor, and every one equal to it
    return launch_pick(residual, start, end, out_idx, out_val,
                       PickRule{nullptr, key_floor, static_cast<int64_t>(0x7FFFFFFFFFFFFFFFll)}, counts, stream);
}

}  // namespace micro
