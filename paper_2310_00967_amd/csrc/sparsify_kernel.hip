// gfx950 kernels of MiCRO's per-worker sparsify step (arXiv 2310.00967).
//
// The step streams a worker's partition [start, end) once (Sec. 4.1,
// Sec. 4.2): grad and residual are read (dwordx4 per lane), acc = grad +
// residual is formed (Sec. 2, error feedback), |acc| is tested against
// theta_f, the residual is written back as selected ? +0 : acc (Algorithm 1,
// reset and carry of the local error), and the selected (index, acc) pairs
// are written in index order (Algorithm 1, selection and gathering of the
// accumulated values).
//
// Order-preserving compaction:
//   * per wavefront row: one ballot per element slot and mbcnt give each
//     lane's rank among the selected values before it in the row;
//   * per workgroup: the wavefront row totals go through LDS, giving each
//     row's offset inside the tile and the tile's count;
//   * across workgroups: decoupled look-back over 64-bit status words
//     (count | flag | epoch), one per tile (ticket schedule) or per chunk of
//     tiles (staged schedule).  Wavefront 0 inspects 64 predecessor tiles
//     or 256 predecessor chunks per round with agent-scope atomic loads,
//     which read the memory level shared by all XCDs.  The count and its flag share one word, so relaxed atomics
//     suffice: a reader sees either the whole published word or an older one.
//
// Staged schedule, three kernels; no workgroup of the first and the last ever
//   waits for another:
//   stream_kernel: one 1024-value tile per 256-thread workgroup, one dwordx4
//     per lane and stream, every HBM stream non-temporal.  It ranks the tile's
//     selected values, writes the residual, packs the pairs in LDS and writes
//     them with coalesced stores to the tile's staging slot (kStageCap
//     8-byte (index, value) records), then stores the tile's count.  A tile
//     with more than kStageCap selected values is left untouched and flagged.
//   scan_kernel: one workgroup per chunk of kChunkTiles tiles: a scan of the
//     chunk's tile counts and a decoupled look-back over chunk status words
//     give every tile its output offset; it records the tile where each move
//     piece starts and lists the flagged tiles.  One look-back per million
//     values keeps the cross-XCD round trips off the streaming pass; a
//     predecessor that has not published is recomputed from its tile counts,
//     so chunks need no ticket.
//   move_kernel: a fixed grid redoes the flagged tiles (one wavefront each)
//     and moves the staged pairs to their final places in equal pieces of the
//     merged sequence of tiles and pairs, whatever the clustering of the
//     selection; it also stores the counts into mapped host memory.
//   stream_scan_kernel (fused staged schedule, the default of a single
//     partition): the stream and scan kernels' work in one launch, each chunk
//     workgroup placed two chunks of tiles after its own chunk's tiles (the
//     last ones after all tiles), polling epoch-tagged tile words; the scans
//     run while the stream goes on, and a launch and its drain are saved.
//   HBM traffic beyond the 12 bytes per value of the stream: 16 bytes per
//   selected value (staged write and read) and 8 bytes per 1024 values.
// Sweep: the same three kernels over a table of segments (every partition of
//   a vector with its own threshold, or a full error-feedback pass split at
//   its partition), each tile also reducing the squared norm of its new
//   residual (the local error of Sec. 2) in a fixed order.
// Ticket schedule: a single pass; 4096-value tiles are drawn from a ticket
//   counter in increasing order, so a tile only waits for tiles claimed by
//   running workgroups; the per-tile ticket and look-back round trips cost
//   bandwidth, but one launch beats two for partitions of up to about a
//   million values.
// accumulate_kernel: the error-feedback addition alone, for the part of the
//   vector a full pass does not search.
#include "sparsify_kernel.h"

namespace micro {
namespace {

constexpr int kWaveSize = 64;

constexpr uint64_t kCountMask = 0xffffffffull;
constexpr uint64_t kFlagAggregate = 1ull << 32;
constexpr uint64_t kFlagInclusive = 2ull << 32;
constexpr uint64_t kFlagMask = 3ull << 32;
constexpr int kLookbackDepth = 4;  // chunk status words per lane and chunk look-back round

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// Cross-lane steps on the data-parallel-primitive (DPP) paths of gfx9: row
// shifts inside rows of 16 lanes, then broadcasts of lane 15 and lane 31 to
// the following rows.  A lane whose source lies outside its row, or a row the
// mask leaves out, receives 0, the identity of both operations used here.
// Every lane of the wavefront must be active.
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143, kDppWaveShr1 = 0x138;

__device__ __forceinline__ uint32_t dpp(uint32_t x, int ctrl) {
    switch (ctrl) {  // the control must be a constant of the instruction
        case kDppRowShr1: return __builtin_amdgcn_update_dpp(0u, x, kDppRowShr1, 0xf, 0xf, false);
        case kDppRowShr2: return __builtin_amdgcn_update_dpp(0u, x, kDppRowShr2, 0xf, 0xf, false);
        case kDppRowShr4: return __builtin_amdgcn_update_dpp(0u, x, kDppRowShr4, 0xf, 0xf, false);
        case kDppRowShr8: return __builtin_amdgcn_update_dpp(0u, x, kDppRowShr8, 0xf, 0xf, false);
        case kDppRowBcast15: return __builtin_amdgcn_update_dpp(0u, x, kDppRowBcast15, 0xa, 0xf, false);
        case kDppRowBcast31: return __builtin_amdgcn_update_dpp(0u, x, kDppRowBcast31, 0xc, 0xf, false);
        default: return __builtin_amdgcn_update_dpp(0u, x, kDppWaveShr1, 0xf, 0xf, false);
    }
}

// Inclusive sum / maximum over lanes 0 .. lane of the wavefront.
__device__ __forceinline__ uint32_t wave_inclusive_sum(uint32_t x) {
    x += dpp(x, kDppRowShr1);
    x += dpp(x, kDppRowShr2);
    x += dpp(x, kDppRowShr4);
    x += dpp(x, kDppRowShr8);
    x += dpp(x, kDppRowBcast15);
    x += dpp(x, kDppRowBcast31);
    return x;
}

__device__ __forceinline__ uint32_t wave_inclusive_max(uint32_t x) {
    uint32_t y;
    y = dpp(x, kDppRowShr1);
    x = y > x ? y : x;
    y = dpp(x, kDppRowShr2);
    x = y > x ? y : x;
    y = dpp(x, kDppRowShr4);
    x = y > x ? y : x;
    y = dpp(x, kDppRowShr8);
    x = y > x ? y : x;
    y = dpp(x, kDppRowBcast15);
    x = y > x ? y : x;
    y = dpp(x, kDppRowBcast31);
    x = y > x ? y : x;
    return x;
}

// The value of the lane below (0 in lane 0).
__device__ __forceinline__ uint32_t wave_shift_up1(uint32_t x) { return dpp(x, kDppWaveShr1); }

// Sum over the wavefront, in every lane.
__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
    return __builtin_amdgcn_readlane(wave_inclusive_sum(v), kWaveSize - 1);
}

__device__ __forceinline__ uint64_t load_status(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void store_status(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Look-back by all 64 lanes of one wavefront over the status words of the
// items (tiles or chunks) before `item`: sums their counts back to the nearest
// inclusive prefix and returns the exclusive prefix (uniform).  Callers draw
// their items from a ticket counter, so every earlier item belongs to a
// running workgroup that publishes its count without waiting for later ones:
// the retries end.
__device__ uint32_t lookback(const uint64_t* status, uint32_t item, uint32_t epoch, int lane) {
    const uint64_t tag = static_cast<uint64_t>(epoch) << kEpochShift;
    uint32_t exclusive = 0;
    int64_t top = static_cast<int64_t>(item) - 1;
    for (;;) {
        const int64_t p = top - lane;
        // Positions before item 0 read as an inclusive prefix of zero; item 0
        // itself always publishes an inclusive word, so they are only reached
        // once every real predecessor in the window is published.
        const uint64_t w = (p >= 0) ? load_status(&status[p]) : (tag | kFlagInclusive);
        const bool valid = (w >> kEpochShift) == epoch && (w & kFlagMask) != 0;
        const bool inclusive = valid && (w & kFlagMask) == kFlagInclusive;
        const uint64_t inc_mask = __ballot(inclusive);
        const uint64_t bad_mask = __ballot(!valid);
        // lanes 0 .. first inclusive lane (all 64 when none is inclusive)
        const uint64_t need = inc_mask ? (inc_mask ^ (inc_mask - 1)) : ~0ull;
        if (bad_mask & need) {
            __builtin_amdgcn_s_sleep(1);
            continue;
        }
        const uint32_t v = ((need >> lane) & 1ull) ? static_cast<uint32_t>(w & kCountMask) : 0u;
        exclusive += wave_sum(v);
        if (inc_mask) return exclusive;
        top -= kWaveSize;
    }
}

// Values of one tile in registers: LANES threads, ROWS rows of VEC consecutive
// values per lane; value (row, lane, c) sits at
// base + (row * LANES + lane) * VEC + c, which is also its output order.
template <int VEC, int ROWS, int LANES>
struct Tile {
    static constexpr int kElems = VEC * ROWS * LANES;
    int64_t base;
    bool interior;       // the whole tile lies inside [start, end)
    float v[ROWS][VEC];  // grad, then acc
    float e[ROWS][VEC];  // residual
};

template <int VEC, int ROWS, int LANES>
__device__ __forceinline__ int64_t elem_index(const Tile<VEC, ROWS, LANES>& t, int r, int lane, int c) {
    return t.base + static_cast<int64_t>(r * LANES + lane) * VEC + c;
}

// Issues every load of the tile whose first value has global index `base`
// (a.base plus a multiple of the tile size).  Interior tiles use dwordx4
// (VEC == 4, 16-byte aligned by the choice of a.base) or dword loads,
// non-temporal when NT (each value is read once); tiles that cross start or
// end load element by element inside [start, end) and read 0 elsewhere.
template <int VEC, int ROWS, int LANES, bool NT>
__device__ __forceinline__ void load_tile(const LaunchArgs& a, int64_t base, int lane,
                                          Tile<VEC, ROWS, LANES>& t) {
    using T = Tile<VEC, ROWS, LANES>;
    t.base = base;
    t.interior = t.base >= a.start && t.base + T::kElems <= a.end;
    if (t.interior) {
        if constexpr (VEC == 4) {
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                const f32x4* p = reinterpret_cast<const f32x4*>(a.grad + elem_index(t, r, lane, 0));
                const f32x4 x = __builtin_nontemporal_load(p);
#pragma unroll
                for (int c = 0; c < 4; ++c) t.v[r][c] = x[c];
            }
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                const f32x4* p = reinterpret_cast<const f32x4*>(a.residual + elem_index(t, r, lane, 0));
                const f32x4 x = NT ? __builtin_nontemporal_load(p) : *p;
#pragma unroll
                for (int c = 0; c < 4; ++c) t.e[r][c] = x[c];
            }
        } else {
#pragma unroll
            for (int r = 0; r < ROWS; ++r)
#pragma unroll
                for (int c = 0; c < VEC; ++c)
                    t.v[r][c] = __builtin_nontemporal_load(a.grad + elem_index(t, r, lane, c));
#pragma unroll
            for (int r = 0; r < ROWS; ++r)
#pragma unroll
                for (int c = 0; c < VEC; ++c) {
                    const float* p = a.residual + elem_index(t, r, lane, c);
                    t.e[r][c] = NT ? __builtin_nontemporal_load(p) : *p;
                }
        }
    } else {
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
#pragma unroll
            for (int c = 0; c < VEC; ++c) {
                const int64_t i = elem_index(t, r, lane, c);
                const bool inside = i >= a.start && i < a.end;
                t.v[r][c] = inside ? a.grad[i] : 0.0f;
                t.e[r][c] = inside ? a.residual[i] : 0.0f;
            }
        }
    }
}

// acc = grad + residual (one binary32 add) and the threshold test; values
// outside [start, end) are never selected.  Leaves acc in t.v and returns the
// lane's selection bits: bit r * VEC + c for value (r, lane, c).  HINT: *zero
// receives the selected values whose residual becomes +0, those with
// |acc| >= theta_zero.
template <int VEC, int ROWS, int LANES, bool HINT = false>
__device__ __forceinline__ uint32_t compute_tile(const LaunchArgs& a, int lane, Tile<VEC, ROWS, LANES>& t,
                                                 uint32_t* zero = nullptr) {
    static_assert(VEC * ROWS <= 32, "selection bits");
    uint32_t sel = 0, z = 0;
    float theta_zero = 0.0f;
    if constexpr (HINT) {
        // read with the other arguments, not where the mask is used: a load
        // sunk to its use is a wait of its own in every workgroup
        theta_zero = a.theta_zero;
        asm volatile("" : "+s"(theta_zero));
    }
#pragma unroll
    for (int r = 0; r < ROWS; ++r)
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            const float acc = t.v[r][c] + t.e[r][c];
            t.v[r][c] = acc;
            bool s = __builtin_fabsf(acc) >= a.theta_f;
            if (!t.interior) {
                const int64_t i = elem_index(t, r, lane, c);
                s = s && i >= a.start && i < a.end;
            }
            sel |= static_cast<uint32_t>(s) << (r * VEC + c);
            if constexpr (HINT) z |= static_cast<uint32_t>(__builtin_fabsf(acc) >= theta_zero) << (r * VEC + c);
        }
    if constexpr (HINT) *zero = sel & z;
    return sel;
}

template <int VEC>
__device__ __forceinline__ bool selected(uint32_t sel, int r, int c) {
    return (sel >> (r * VEC + c)) & 1u;
}

// residual = selected ? +0 : acc, inside [start, end) only.
template <int VEC, int ROWS, int LANES, bool NT>
__device__ __forceinline__ void store_residual(const LaunchArgs& a, int lane, const Tile<VEC, ROWS, LANES>& t,
                                               uint32_t sel) {
    if (t.interior) {
        if constexpr (VEC == 4) {
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                f32x4 out;
#pragma unroll
                for (int c = 0; c < 4; ++c) out[c] = selected<4>(sel, r, c) ? 0.0f : t.v[r][c];
                f32x4* p = reinterpret_cast<f32x4*>(a.residual + elem_index(t, r, lane, 0));
                if (NT)
                    __builtin_nontemporal_store(out, p);
                else
                    *p = out;
            }
        } else {
#pragma unroll
            for (int r = 0; r < ROWS; ++r)
#pragma unroll
                for (int c = 0; c < VEC; ++c) {
                    float* p = a.residual + elem_index(t, r, lane, c);
                    const float out = selected<VEC>(sel, r, c) ? 0.0f : t.v[r][c];
                    if (NT)
                        __builtin_nontemporal_store(out, p);
                    else
                        *p = out;
                }
        }
    } else {
#pragma unroll
        for (int r = 0; r < ROWS; ++r)
#pragma unroll
            for (int c = 0; c < VEC; ++c) {
                const int64_t i = elem_index(t, r, lane, c);
                if (i >= a.start && i < a.end) a.residual[i] = selected<VEC>(sel, r, c) ? 0.0f : t.v[r][c];
            }
    }
}

// Ranks of a wavefront's selected values: lane_rank[r] = number of selected
// values before the lane's first value of row r among the wavefront's values
// of that row; row_count[r] = the wavefront's count in row r (uniform).
template <int VEC, int ROWS>
__device__ __forceinline__ void wave_ranks(uint32_t sel, uint32_t (&lane_rank)[ROWS],
                                           uint32_t (&row_count)[ROWS]) {
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        uint32_t below = 0, total = 0;
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            const uint64_t m = __ballot(selected<VEC>(sel, r, c));
            below += lanes_below(m);
            total += static_cast<uint32_t>(__popcll(m));
        }
        lane_rank[r] = below;
        row_count[r] = total;
    }
}

// Workgroup-level ranks: each wavefront's row counts go through LDS (the
// wavefront parts of a row are ordered by wavefront, rows by row);
// row_base[r] receives this wavefront's offset of row r inside the tile and
// the tile's count is returned.  Contains one barrier.
template <int ROWS, int WAVES>
__device__ __forceinline__ uint32_t tile_ranks(const uint32_t (&row_count)[ROWS], int lane, int wave,
                                               uint32_t* s_wave_total, uint32_t (&row_base)[ROWS]) {
    if (lane == 0) {
#pragma unroll
        for (int r = 0; r < ROWS; ++r) s_wave_total[r * WAVES + wave] = row_count[r];
    }
    __syncthreads();
    uint32_t running = 0;
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
#pragma unroll
        for (int w = 0; w < WAVES; ++w) {
            const uint32_t v = s_wave_total[r * WAVES + w];
            if (w == wave) row_base[r] = running;
            running += v;
        }
    }
    return running;
}

// Writes the selected (index, acc) pairs: the k-th selected value of row r of
// this lane goes to position out_base + row_base[r] + lane_rank[r] + k.
template <int VEC, int ROWS, int LANES>
__device__ __forceinline__ void scatter_pairs(const LaunchArgs& a, int lane, const Tile<VEC, ROWS, LANES>& t,
                                              uint32_t sel, uint32_t out_base, const uint32_t (&row_base)[ROWS],
                                              const uint32_t (&lane_rank)[ROWS]) {
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        uint32_t pos = out_base + row_base[r] + lane_rank[r];
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            if (selected<VEC>(sel, r, c)) {
                a.out_idx[pos] = static_cast<int32_t>(elem_index(t, r, lane, c));
                a.out_val[pos] = t.v[r][c];
                ++pos;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Staged schedule
// ---------------------------------------------------------------------------

constexpr uint32_t kOverflow = 0x80000000u;
constexpr int kMoveBatch = 8;      // independent copies in flight per thread
constexpr int kWindowBatch = 8;    // window loads in flight per thread
// s_waitcnt operand (gfx9 encoding): vector-memory count 0, export and
// LDS/scalar-memory counts at their maxima (not waited for)
constexpr int kWaitVmcnt0 = 0x0F70;

// Draws the workgroup's ticket (thread 0) and rearms the counter when the
// last ticket of the launch is drawn: every other workgroup of the launch has
// drawn its ticket by then.
__device__ __forceinline__ uint32_t draw_ticket(unsigned long long* counter, uint32_t last) {
    const uint32_t drawn = static_cast<uint32_t>(atomicAdd(counter, 1ull));
    if (drawn == last) __hip_atomic_store(counter, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return drawn;
}

// Segment of a sweep holding global tile `tile` (or scan chunk `chunk`): the
// last segment whose first tile (chunk) is <= it, so empty segments are
// skipped.  Uniform binary search over the table in the kernel arguments.
__device__ __forceinline__ uint32_t segment_of_tile(const SweepTable* tbl, uint32_t tile) {
    uint32_t lo = 0, hi = tbl->count;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) / 2;
        if (tbl->seg[mid].tile_first <= tile)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

__device__ __forceinline__ uint32_t segment_of_chunk(const SweepTable* tbl, uint32_t chunk) {
    uint32_t lo = 0, hi = tbl->count;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) / 2;
        if (tbl->seg[mid].chunk_first <= chunk)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

// A sweep segment's range and threshold in the fields the tile helpers read;
// returns the global index of the first value of the segment's tile `tile`.
__device__ __forceinline__ int64_t enter_segment(LaunchArgs& a, const SweepTable* tbl, uint32_t tile) {
    const SweepSegment& sg = tbl->seg[segment_of_tile(tbl, tile)];
    a.start = sg.start;
    a.end = sg.end;
    a.theta_f = sg.theta_f;
    return sg.base + static_cast<int64_t>(tile - sg.tile_first) * kStreamTile;
}

// Sum over the workgroup of one binary64 value per thread, in a fixed order
// (a butterfly inside each wavefront, then the wavefronts in order); the
// result is valid in thread 0.  Contains one barrier.
template <int WAVES>
__device__ __forceinline__ double block_sum(double v, int lane, int wave, double* s_part) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWaveSize);
    if (lane == 0) s_part[wave] = v;
    __syncthreads();
    double total = 0.0;
    if (wave == 0 && lane == 0) {
#pragma unroll
        for (int w = 0; w < WAVES; ++w) total += s_part[w];
    }
    return total;
}

// A tile's count (bit 31: left to the move kernel): a plain word for the scan
// kernel of the next launch or, in the fused schedule, an epoch-tagged status
// word that the chunk workgroups of the same launch poll.
template <bool FUSED>
__device__ __forceinline__ void publish_tile(const LaunchArgs& a, uint32_t tile, uint32_t raw) {
    if constexpr (FUSED)
        store_status(&a.tile_words[tile], (static_cast<uint64_t>(a.epoch) << kEpochShift) | kFlagAggregate | raw);
    else
        a.tile_counts[tile] = raw;
}

// Stream pass over one tile (see the file comment).  In a sweep the tile's
// segment supplies range and threshold, and the tile also stores the squared
// norm of its new residual (also for a tile left to the move kernel, whose
// new residual is fixed by its selection bits all the same).
template <int VEC, int ROWS, bool SWEEP, bool FUSED = false, bool HINT = false>
__device__ __forceinline__ void stream_tile(LaunchArgs a, const SweepTable* tbl, uint32_t tile) {
    constexpr int WAVES = kStreamBlock / kWaveSize;
    static_assert(VEC * ROWS * kStreamBlock == kStreamTile, "tile size");
    __shared__ uint32_t s_wave_total[ROWS * WAVES];
    __shared__ uint2 s_pair[kStageCap];  // (index, value bits)
    __shared__ double s_sq[WAVES];

    const int tid = threadIdx.x;
    const int lane = tid & (kWaveSize - 1);
    const int wave = tid / kWaveSize;
    const int64_t tile_base = SWEEP ? enter_segment(a, tbl, tile) : a.base + static_cast<int64_t>(tile) * kStreamTile;

    Tile<VEC, ROWS, kStreamBlock> t;
    uint32_t lane_rank[ROWS], row_count[ROWS], row_base[ROWS];
    load_tile<VEC, ROWS, kStreamBlock, true>(a, tile_base, tid, t);
    uint32_t zero = 0;
    const uint32_t sel = compute_tile<VEC, ROWS, kStreamBlock, HINT>(a, tid, t, &zero);
    if constexpr (SWEEP) {
        double sq = 0.0;
#pragma unroll
        for (int r = 0; r < ROWS; ++r)
#pragma unroll
            for (int c = 0; c < VEC; ++c) {
                const int64_t i = elem_index(t, r, tid, c);
                const double v = selected<VEC>(sel, r, c) ? 0.0 : static_cast<double>(t.v[r][c]);
                if (i >= a.start && i < a.end) sq += v * v;
            }
        const double total = block_sum<WAVES>(sq, lane, wave, s_sq);
        if (tid == 0) a.tile_sumsq[tile] = total;
    }
    wave_ranks<VEC, ROWS>(sel, lane_rank, row_count);
    const uint32_t count = tile_ranks<ROWS, WAVES>(row_count, lane, wave, s_wave_total, row_base);
    if (count > kStageCap) {  // uniform: left to the move kernel, residual untouched
        if (tid == 0) publish_tile<FUSED>(a, tile, count | kOverflow);
        return;
    }
    store_residual<VEC, ROWS, kStreamBlock, true>(a, tid, t, HINT ? zero : sel);
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        uint32_t pos = row_base[r] + lane_rank[r];
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            if (selected<VEC>(sel, r, c)) {
                s_pair[pos] = make_uint2(static_cast<uint32_t>(elem_index(t, r, tid, c)),
                                         __float_as_uint(t.v[r][c]));
                ++pos;
            }
        }
    }
    __syncthreads();
    uint64_t* slot = reinterpret_cast<uint64_t*>(a.stage) + static_cast<size_t>(tile) * kStageCap;
    for (uint32_t j = tid; j < count; j += kStreamBlock) {
        const uint2 p = s_pair[j];  // index in the low word, value bits in the high word
        __builtin_nontemporal_store(static_cast<uint64_t>(p.x) | (static_cast<uint64_t>(p.y) << 32), slot + j);
    }
    if (tid == 0) publish_tile<FUSED>(a, tile, count);
}

template <int VEC, int ROWS>
__global__ __launch_bounds__(kStreamBlock) void stream_kernel(LaunchArgs a) {
    stream_tile<VEC, ROWS, false>(a, nullptr, blockIdx.x);
}

// The stream pass that sets only the residual of values at or above
// theta_zero to +0.
template <int VEC, int ROWS>
__global__ __launch_bounds__(kStreamBlock) void stream_hint_kernel(LaunchArgs a) {
    stream_tile<VEC, ROWS, false, false, true>(a, nullptr, blockIdx.x);
}

template <int VEC, int ROWS>
__global__ __launch_bounds__(kStreamBlock) void stream_sweep_kernel(LaunchArgs a, SweepTable tbl) {
    stream_tile<VEC, ROWS, true>(a, &tbl, blockIdx.x);
}

// Full processing of one flagged tile by one wavefront with its pairs from
// position out_base on: the tile's values in index order, 256 at a time (one
// part in registers keeps the move kernel's register budget).  a carries the
// tile's range and threshold; tile_base is its first value's global index.
template <int VEC, bool HINT = false>
__device__ void redo_tile(const LaunchArgs& a, int64_t tile_base, int lane, uint32_t out_base) {
    constexpr int ROWS = 4 / VEC;
    using T = Tile<VEC, ROWS, kWaveSize>;
    static_assert(kStreamTile % T::kElems == 0, "whole parts");
    uint32_t run = out_base;
#pragma unroll 1
    for (int part = 0; part < kStreamTile / T::kElems; ++part) {
        T t;
        uint32_t lane_rank[ROWS], row_count[ROWS], row_base[ROWS];
        load_tile<VEC, ROWS, kWaveSize, false>(a, tile_base + part * T::kElems, lane, t);
        uint32_t zero = 0;
        const uint32_t sel = compute_tile<VEC, ROWS, kWaveSize, HINT>(a, lane, t, &zero);
        wave_ranks<VEC, ROWS>(sel, lane_rank, row_count);
        uint32_t sub = 0;
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
            row_base[r] = sub;
            sub += row_count[r];
        }
        store_residual<VEC, ROWS, kWaveSize, false>(a, lane, t, HINT ? zero : sel);
        scatter_pairs(a, lane, t, sel, run, row_base, lane_rank);
        run += sub;
    }
}

// The flagged-tile counter count_out[1] holds (epoch << 32) | count; a word
// of an older launch reads as zero, so it is never cleared between launches.
// reserve_flagged adds n for this launch and returns the first list position
// of the n entries (one compare-and-swap loop per chunk that has flagged
// tiles; those are rare).
__device__ __forceinline__ uint32_t reserve_flagged(const LaunchArgs& a, uint32_t n) {
    unsigned long long* p = reinterpret_cast<unsigned long long*>(&a.count_out[1]);
    unsigned long long old = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (;;) {
        const uint32_t base = (old >> 32) == a.epoch ? static_cast<uint32_t>(old) : 0u;
        const unsigned long long next = (static_cast<unsigned long long>(a.epoch) << 32) | (base + n);
        const unsigned long long seen = atomicCAS(p, old, next);
        if (seen == old) return base;
        old = seen;
    }
}

// This launch's flagged-tile count from the counter word.
__device__ __forceinline__ uint32_t flagged_count(const LaunchArgs& a, int64_t word) {
    const uint64_t w = static_cast<uint64_t>(word);
    return (w >> 32) == a.epoch ? static_cast<uint32_t>(w) : 0u;
}

// Tiles [first, end) of scan chunk `chunk`: kChunkTiles per chunk; in a
// sweep each segment has chunks of its own, the last one possibly short.
template <bool SWEEP>
__device__ __forceinline__ void chunk_tiles(const LaunchArgs& a, const SweepTable* tbl, uint32_t chunk,
                                            uint32_t& first, uint32_t& end) {
    if constexpr (SWEEP) {
        const uint32_t r = segment_of_chunk(tbl, chunk);
        first = tbl->seg[r].tile_first + (chunk - tbl->seg[r].chunk_first) * kChunkTiles;
        const uint32_t seg_end = tbl->seg[r + 1].tile_first;
        end = first + kChunkTiles < seg_end ? first + kChunkTiles : seg_end;
    } else {
        first = chunk * kChunkTiles;
        end = first + kChunkTiles < a.num_tiles ? first + kChunkTiles : a.num_tiles;
    }
}

// The counts of N tiles (bit 31: left to the move kernel) of the fused
// schedule, t[i] < end only (others read 0): their epoch-tagged words are
// loaded together and the ones not yet published polled again.  Only stream
// workgroups publish tile words and they wait for nobody, so the loop ends.
template <int N>
__device__ __forceinline__ void poll_tiles(const LaunchArgs& a, const uint32_t (&t)[N], uint32_t end,
                                           uint32_t (&raw)[N]) {
    uint32_t pending = 0;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        raw[i] = 0;
        if (t[i] < end) pending |= 1u << i;
    }
    while (pending) {
        uint64_t w[N];
#pragma unroll
        for (int i = 0; i < N; ++i) w[i] = (pending >> i) & 1u ? load_status(&a.tile_words[t[i]]) : 0ull;
#pragma unroll
        for (int i = 0; i < N; ++i) {
            if (((pending >> i) & 1u) && (w[i] >> kEpochShift) == a.epoch && (w[i] & kFlagMask) != 0) {
                raw[i] = static_cast<uint32_t>(w[i] & kCountMask);
                pending &= ~(1u << i);
            }
        }
        if (pending) __builtin_amdgcn_s_sleep(2);
    }
}

// poll_tiles for wavefront 0 of a fused chunk workgroup, which also reloads
// the look-back's first window of chunk status words (lane l, slot j: chunk
// - 1 - (l * kLookbackDepth + j); before chunk 0 an inclusive zero) in every
// round, until no lane of the wavefront waits for a tile.  win receives the
// lane's words of the last round: by the time a chunk's last tile is in, the
// chunk before it has usually published, so the look-back often needs no
// round trip of its own.
template <int N>
__device__ __forceinline__ void poll_tiles_and_window(const LaunchArgs& a, const uint32_t (&t)[N], uint32_t end,
                                                      uint32_t (&raw)[N], uint32_t chunk, int lane,
                                                      uint64_t (&win)[kLookbackDepth]) {
    const uint64_t before_first = (static_cast<uint64_t>(a.epoch) << kEpochShift) | kFlagInclusive;
    uint32_t pending = 0;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        raw[i] = 0;
        if (t[i] < end) pending |= 1u << i;
    }
    for (;;) {  // uniform across the wavefront
        uint64_t w[N];
#pragma unroll
        for (int i = 0; i < N; ++i) w[i] = (pending >> i) & 1u ? load_status(&a.tile_words[t[i]]) : 0ull;
#pragma unroll
        for (int j = 0; j < kLookbackDepth; ++j) {
            const int64_t p = static_cast<int64_t>(chunk) - 1 - (lane * kLookbackDepth + j);
            win[j] = p >= 0 ? load_status(&a.chunk_status[p]) : before_first;
        }
#pragma unroll
        for (int i = 0; i < N; ++i) {
            if (((pending >> i) & 1u) && (w[i] >> kEpochShift) == a.epoch && (w[i] & kFlagMask) != 0) {
                raw[i] = static_cast<uint32_t>(w[i] & kCountMask);
                pending &= ~(1u << i);
            }
        }
        if (__ballot(pending != 0) == 0) return;
        __builtin_amdgcn_s_sleep(2);
    }
}

// Selected values of chunk `chunk`, summed from its tile counts by one
// wavefront (uniform): the count the chunk's own workgroup publishes.
template <bool SWEEP>
__device__ uint32_t chunk_selected(const LaunchArgs& a, const SweepTable* tbl, uint32_t chunk, int lane) {
    uint32_t first, end;
    chunk_tiles<SWEEP>(a, tbl, chunk, first, end);
    uint32_t v = 0;
#pragma unroll
    for (int i = 0; i < kChunkTiles / kWaveSize; ++i) {
        const uint32_t t = first + i * kWaveSize + lane;
        v += t < end ? (a.tile_counts[t] & ~kOverflow) : 0u;
    }
    return wave_sum(v);
}

constexpr int kLookbackPolls = 4;  // polls of a silent predecessor before its count is recomputed

// Exclusive prefix of chunk `chunk`: a look-back by all 64 lanes of one
// wavefront over the status words of the chunks before it, back to the
// nearest inclusive prefix.  Chunks are not handed out in order (no ticket),
// so a predecessor may not have run yet: a word still unpublished after a few
// polls is replaced by the predecessor's count summed from its tile counts,
// which are final before the scan kernel starts.  The look-back therefore
// ends whatever order the workgroups run in.  In the fused schedule a
// predecessor's tile words may still be missing, so a recompute would have to
// wait for them anyway: there the look-back polls until each predecessor has
// published (a chunk workgroup publishes its aggregate as soon as its tile
// words are in, before its own look-back, so the wait depends on stream
// workgroups only, and its predecessors sit at lower indices of the launch).
// Each round a lane reads kLookbackDepth words, so a round covers 256
// predecessors (the GPT-1.3B partition's 1,285 chunks need at most six
// rounds instead of twenty-one).  In the fused schedule `first` holds the
// lane's words of the first window, read while the chunk's tile words were
// polled (older observations of the same words, which the look-back treats
// like any other poll).
template <bool SWEEP, bool FUSED = false>
__device__ uint32_t chunk_lookback(const LaunchArgs& a, const SweepTable* tbl, uint32_t chunk, int lane,
                                   const uint64_t (&first)[kLookbackDepth]) {
    constexpr int D = kLookbackDepth;
    const uint64_t tag = static_cast<uint64_t>(a.epoch) << kEpochShift;
    uint32_t exclusive = 0;
    int64_t top = static_cast<int64_t>(chunk) - 1;
    int polls = 0;
    bool have_first = FUSED;
    for (;;) {
        // slot j of lane l holds predecessor top - (l * D + j): the window's
        // nearest word is lane 0's slot 0; positions before chunk 0 read as
        // an inclusive prefix of zero
        uint64_t w[D];
        uint32_t valid_bits = 0, incl_bits = 0;
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const int64_t p = top - (lane * D + j);
            w[j] = have_first ? first[j] : (p >= 0) ? load_status(&a.chunk_status[p]) : (tag | kFlagInclusive);
        }
        have_first = false;
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const bool valid = (w[j] >> kEpochShift) == a.epoch && (w[j] & kFlagMask) != 0;
            valid_bits |= static_cast<uint32_t>(valid) << j;
            incl_bits |= static_cast<uint32_t>(valid && (w[j] & kFlagMask) == kFlagInclusive) << j;
        }
        const uint64_t inc_lanes = __ballot(incl_bits != 0);
        const int first_lane = inc_lanes ? __builtin_ctzll(inc_lanes) : kWaveSize;  // uniform
        // the slots up to the nearest inclusive word (all of them when there is none)
        const uint32_t need_bits = lane < first_lane    ? (1u << D) - 1u
                                   : lane == first_lane ? (2u << __builtin_ctz(incl_bits)) - 1u
                                                        : 0u;
        const uint32_t miss_bits = need_bits & ~valid_bits;
        const bool missing = __ballot(miss_bits != 0) != 0;  // uniform
        if (missing && (FUSED || ++polls < kLookbackPolls)) {
            __builtin_amdgcn_s_sleep(1);
            continue;
        }
        polls = 0;
        uint32_t v = 0;
#pragma unroll
        for (int j = 0; j < D; ++j)
            if (((need_bits & valid_bits) >> j) & 1u) v += static_cast<uint32_t>(w[j] & kCountMask);
        if (missing) {  // uniform: sum each missing predecessor from its tile counts
#pragma unroll 1
            for (int j = 0; j < D; ++j) {
                uint64_t m = __ballot((miss_bits >> j) & 1u);
                while (m) {
                    const int l = __builtin_ctzll(m);
                    m &= m - 1;
                    const uint32_t c = chunk_selected<SWEEP>(a, tbl, static_cast<uint32_t>(top - (l * D + j)), lane);
                    if (lane == l) v += c;
                }
            }
        }
        exclusive += wave_sum(v);
        if (inc_lanes) return exclusive;
        top -= kWaveSize * D;
    }
}

// Scan kernel: one workgroup per chunk of kChunkTiles tiles (chunk =
// workgroup index).  Scans the chunk's tile counts, finds the chunk's output
// offset by decoupled look-back over chunk status words (chunk_lookback), publishes every tile's output offset
// (bit 31: flagged tile), records for every move piece the tile that holds
// its first item, and appends the chunk's flagged tiles to the list that the
// move kernel redoes.
// In a sweep the chunk lies inside one segment (chunks never straddle two)
// and also sums its tiles' squared norms; the look-back and the offsets are
// global, since the segments' pairs form one compaction in index order.
// FUSED: the same work by the chunk workgroups of stream_scan_kernel, which
// poll their chunk's epoch-tagged tile words instead of reading final counts.
template <bool SWEEP, bool FUSED = false>
__device__ __forceinline__ void scan_chunk(const LaunchArgs& a, const SweepTable* tbl, uint32_t chunk) {
    constexpr int WAVES = kScanBlock / kWaveSize;
    constexpr int PER_THREAD = kChunkTiles / kScanBlock;
    static_assert(PER_THREAD % 4 == 0, "whole uint4s of counts per thread");
    __shared__ uint32_t s_exclusive, s_num_flagged, s_list_base;
    __shared__ uint32_t s_wave_total[WAVES];
    __shared__ uint32_t s_flagged[kChunkTiles];

    const int tid = threadIdx.x;
    const int lane = tid & (kWaveSize - 1);
    const int wave = tid / kWaveSize;
    if (tid == 0) s_num_flagged = 0;
    uint32_t chunk_tile, end_tile;
    chunk_tiles<SWEEP>(a, tbl, chunk, chunk_tile, end_tile);
    const uint32_t first_tile = chunk_tile + tid * PER_THREAD;
    const bool whole = first_tile % 4 == 0 && first_tile + PER_THREAD <= end_tile;

    uint32_t raw[PER_THREAD];
    uint64_t window[kLookbackDepth] = {};  // fused schedule, wave 0: the look-back's first window
    if constexpr (FUSED) {
        uint32_t t[PER_THREAD];
#pragma unroll
        for (int i = 0; i < PER_THREAD; ++i) t[i] = first_tile + i;
        if (wave == 0)
            poll_tiles_and_window<PER_THREAD>(a, t, end_tile, raw, chunk, lane, window);
        else
            poll_tiles<PER_THREAD>(a, t, end_tile, raw);
    } else if (whole) {
#pragma unroll
        for (int i = 0; i < PER_THREAD; i += 4) {
            const uint4 v = *reinterpret_cast<const uint4*>(a.tile_counts + first_tile + i);
            raw[i] = v.x;
            raw[i + 1] = v.y;
            raw[i + 2] = v.z;
            raw[i + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < PER_THREAD; ++i) raw[i] = first_tile + i < end_tile ? a.tile_counts[first_tile + i] : 0u;
    }
    uint32_t mine = 0;
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) mine += raw[i] & ~kOverflow;
    const uint32_t x = wave_inclusive_sum(mine);  // inclusive scan of thread totals inside the wavefront
    if (lane == kWaveSize - 1) s_wave_total[wave] = x;
    __syncthreads();
    uint32_t before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
        if (w < wave) before += s_wave_total[w];
        total += s_wave_total[w];
    }
    if (wave == 0) {
        const uint64_t tag = static_cast<uint64_t>(a.epoch) << kEpochShift;
        uint32_t excl = 0;
        if (chunk == 0) {
            if (lane == 0) store_status(&a.chunk_status[0], tag | kFlagInclusive | total);
        } else {
            if (lane == 0) store_status(&a.chunk_status[chunk], tag | kFlagAggregate | total);
            excl = chunk_lookback<SWEEP, FUSED>(a, tbl, chunk, lane, window);
            if (lane == 0) store_status(&a.chunk_status[chunk], tag | kFlagInclusive | (excl + total));
        }
        if (lane == 0) {
            s_exclusive = excl;
            if (chunk == a.num_chunks - 1) a.count_out[0] = static_cast<int64_t>(excl) + total;
        }
    }
    __syncthreads();
    uint32_t pos = s_exclusive + before + x - mine;  // output offset of my first tile
    const uint32_t span_shift = 31 - __builtin_clz(a.move_span);  // a power of two
    uint32_t offs[PER_THREAD];
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
        const uint32_t count = raw[i] & ~kOverflow;
        offs[i] = pos | (raw[i] & kOverflow);
        // The move pieces whose first item falls among this tile's items: the
        // tile's own item sits at tile + pos in the merged sequence and its
        // count pairs follow it.  A tile spans up to kStreamTile + 1 items,
        // so with pieces of kStreamTile items or fewer it can hold several
        // pieces' first items (at most three with 512-item pieces).
        if (first_tile + i < end_tile) {
            const uint64_t item = static_cast<uint64_t>(first_tile + i) + pos;
            const uint64_t end_item = item + 1 + count;
            for (uint64_t m = (item + a.move_span - 1) >> span_shift; (m << span_shift) < end_item; ++m)
                a.split_tile[m] = first_tile + i;
        }
        if (raw[i] & kOverflow) s_flagged[atomicAdd(&s_num_flagged, 1u)] = first_tile + i;
        pos += count;
    }
    if (whole) {
#pragma unroll
        for (int i = 0; i < PER_THREAD; i += 4)
            *reinterpret_cast<uint4*>(a.tile_excl + first_tile + i) =
                make_uint4(offs[i], offs[i + 1], offs[i + 2], offs[i + 3]);
    } else {
#pragma unroll
        for (int i = 0; i < PER_THREAD; ++i)
            if (first_tile + i < end_tile) a.tile_excl[first_tile + i] = offs[i];
    }
    __syncthreads();
    const uint32_t flagged = s_num_flagged;
    if (flagged == 0) return;  // uniform
    if (tid == 0) s_list_base = reserve_flagged(a, flagged);
    __syncthreads();
    for (uint32_t f = tid; f < flagged; f += kScanBlock) a.flagged_list[s_list_base + f] = s_flagged[f];
}

__global__ __launch_bounds__(kScanBlock) void scan_kernel(LaunchArgs a) { scan_chunk<false>(a, nullptr, blockIdx.x); }

// Fused schedule: workgroups [0, num_tiles) stream the tiles (stream_kernel's
// work, publishing epoch-tagged tile words), workgroups [num_tiles,
// num_tiles + num_chunks) scan the chunks (scan_kernel's work, polling the
// tile words of their chunk).
// Forward progress rests on two facts.  (1) Every wait targets a workgroup of
// lower index in the same launch: a chunk workgroup waits for the tile words
// of its own chunk (stream workgroups, which wait for nobody) and, in its
// look-back, for the aggregates of lower chunks (each published as soon as
// that chunk's tile words are in, before its own look-back).  (2) Each XCD
// dispatches its share of the grid in increasing workgroup index, so a
// workgroup is dispatched once the lower-index workgroups of the launch on
// its XCD have freed a slot.  By induction on the index, the lowest
// unfinished workgroup of the launch is always dispatched eventually and
// never waits for an unfinished one, so every wait ends.  Since each chunk
// workgroup follows its own chunk's tiles by two chunks of tiles (fused_role),
// it mostly finds them published, and at any moment only the few whose tiles
// are still finishing poll, so they hold a negligible share of the slots that
// other resident work could need.
template <int VEC, int ROWS>
__global__ __launch_bounds__(kStreamBlock) void stream_scan_kernel(LaunchArgs a) {
    static_assert(kStreamBlock == kScanBlock, "one workgroup size for both parts");
    const FusedRole role = fused_role(blockIdx.x, a.num_tiles, a.num_chunks);
    if (role.scan)
        scan_chunk<false, true>(a, nullptr, role.item);
    else
        stream_tile<VEC, ROWS, false, true>(a, nullptr, role.item);
}

// The fused launch whose stream pass sets only the residual of values at or
// above theta_zero to +0.
template <int VEC, int ROWS>
__global__ __launch_bounds__(kStreamBlock) void stream_scan_hint_kernel(LaunchArgs a) {
    static_assert(kStreamBlock == kScanBlock, "one workgroup size for both parts");
    const FusedRole role = fused_role(blockIdx.x, a.num_tiles, a.num_chunks);
    if (role.scan)
        scan_chunk<false, true>(a, nullptr, role.item);
    else
        stream_tile<VEC, ROWS, false, true, true>(a, nullptr, role.item);
}

__global__ __launch_bounds__(kScanBlock) void scan_sweep_kernel(LaunchArgs a, SweepTable tbl) {
    scan_chunk<true>(a, &tbl, blockIdx.x);
}

// Segment of a fused sweep holding workgroup b: the last segment whose first
// workgroup is <= b, so empty segments are skipped.  Uniform binary search
// over the table in the kernel arguments.
__device__ __forceinline__ uint32_t segment_of_workgroup(const SweepTable* tbl, uint32_t b) {
    uint32_t lo = 0, hi = tbl->count;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) / 2;
        if (tbl->seg[mid].wg_first <= b)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

// Fused sweep: the stream and scan passes of every segment in one launch.
// Each segment's workgroups follow the previous segment's and are laid out
// like a single partition's fused launch, so every scan workgroup still comes
// after its chunk's tiles and after the scan workgroups of all lower chunks,
// which is all the look-back waits for.
template <int VEC, int ROWS>
__global__ __launch_bounds__(kStreamBlock) void stream_scan_sweep_kernel(LaunchArgs a, SweepTable tbl) {
    static_assert(kStreamBlock == kScanBlock, "one workgroup size for both parts");
    const uint32_t r = segment_of_workgroup(&tbl, blockIdx.x);
    const SweepSegment& sg = tbl.seg[r];
    const SweepSegment& next = tbl.seg[r + 1];
    const FusedRole role = fused_role(blockIdx.x - sg.wg_first, next.tile_first - sg.tile_first,
                                      next.chunk_first - sg.chunk_first);
    if (role.scan)
        scan_chunk<true, true>(a, &tbl, sg.chunk_first + role.item);
    else
        stream_tile<VEC, ROWS, true, true>(a, &tbl, sg.tile_first + role.item);
}

// Number of output pairs before item x of the merged sequence, given the tile
// t whose items contain x and its output offset off: the tile's own item sits
// at t + off and its pairs follow it.
__device__ __forceinline__ uint32_t pairs_before(uint64_t x, uint32_t t, uint32_t off) {
    const uint64_t item = static_cast<uint64_t>(t) + off;
    return off + (x > item ? static_cast<uint32_t>(x - item - 1) : 0u);
}

// Inclusive running maximum over v[0, kMoveSpan) by the whole workgroup: each
// thread takes 16 consecutive entries, read and written as two 16-byte words
// (v is 16-byte aligned).  Contains two barriers; the caller synchronises
// before the entries are read.
__device__ __forceinline__ void block_max_scan(uint16_t* v, int tid, uint32_t* s_wave_max) {
    static_assert(kMoveSpan == 16 * kMoveBlock, "16 entries per thread");
    const int lane = tid & (kWaveSize - 1);
    const int wave = tid / kWaveSize;
    uint4* p = reinterpret_cast<uint4*>(v) + 2 * tid;
    const uint4 w0 = p[0], w1 = p[1];
    uint32_t w[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {  // two entries per word, the lower one first
        const uint32_t e0 = w[i] & 0xffffu, e1 = w[i] >> 16;
        m = e0 > m ? e0 : m;
        const uint32_t r0 = m;
        m = e1 > m ? e1 : m;
        w[i] = r0 | (m << 16);
    }
    const uint32_t incl = wave_inclusive_max(m);  // over the threads of the wavefront
    uint32_t before = wave_shift_up1(incl);
    if (lane == kWaveSize - 1) s_wave_max[wave] = incl;
    __syncthreads();
    for (int k = 0; k < wave; ++k) before = s_wave_max[k] > before ? s_wave_max[k] : before;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        uint32_t e0 = w[i] & 0xffffu, e1 = w[i] >> 16;
        e0 = e0 > before ? e0 : before;
        e1 = e1 > before ? e1 : before;
        w[i] = e0 | (e1 << 16);
    }
    p[0] = make_uint4(w[0], w[1], w[2], w[3]);
    p[1] = make_uint4(w[4], w[5], w[6], w[7]);
    __syncthreads();
}

// The move kernel's work once the count k > 0 is known: the flagged tiles,
// then this workgroup's pieces (first_t0 / first_t1: the split words of its
// first piece, loaded with the counts).
template <int VEC, bool SWEEP, bool HINT = false>
__device__ __forceinline__ void move_work(const LaunchArgs& a, const SweepTable* tbl, int64_t k, uint32_t flagged,
                                          uint32_t first_t0, uint32_t first_t1) {
    constexpr uint32_t kWindow = kMoveSpan + 1;
    constexpr int WAVES = kMoveBlock / kWaveSize;
    static_assert(kWindow <= 65536, "window indices fit in 16 bits");
    __shared__ uint32_t s_off[kWindow];
    __shared__ uint32_t s_flag_bits[(kWindow + 31) / 32];
    __shared__ __align__(16) uint16_t s_owner[kMoveSpan];
    __shared__ uint32_t s_wave_max[WAVES];
    const int tid = threadIdx.x;
    const int lane = tid & (kWaveSize - 1);
    // Flagged tiles first, one wavefront each over the whole grid: the
    // wavefront recomputes the tile and writes its pairs and residual.
    for (uint32_t f = blockIdx.x * WAVES + tid / kWaveSize; f < flagged; f += gridDim.x * WAVES) {
        const uint32_t tile = a.flagged_list[f];
        const uint32_t out_base = a.tile_excl[tile] & ~kOverflow;
        if constexpr (SWEEP) {
            LaunchArgs seg_args = a;
            const int64_t tile_base = enter_segment(seg_args, tbl, tile);
            redo_tile<VEC>(seg_args, tile_base, lane, out_base);
        } else {
            redo_tile<VEC, HINT>(a, a.base + static_cast<int64_t>(tile) * kStreamTile, lane, out_base);
        }
    }
    const uint64_t total = static_cast<uint64_t>(a.num_tiles) + static_cast<uint64_t>(k);
    const uint32_t span_items = a.move_span < kMoveSpan ? a.move_span : kMoveSpan;
    const uint32_t span_shift = 31 - __builtin_clz(span_items);  // a power of two
    const uint32_t pieces = static_cast<uint32_t>((total + span_items - 1) >> span_shift);
    for (uint32_t m = blockIdx.x; m < pieces; m += gridDim.x) {
        const bool first = m == blockIdx.x;
        const uint32_t t0 = first ? first_t0 : a.split_tile[m];
        const uint32_t t1 = m + 1 < pieces ? (first ? first_t1 : a.split_tile[m + 1]) : a.num_tiles - 1;
        // t1 - t0 <= span_items by construction; the clamp only keeps LDS
        // accesses inside the window
        const uint32_t span = t1 - t0 + 1;
        const uint32_t ntiles = span < kWindow ? span : kWindow;
        for (uint32_t i = tid; i < (ntiles + 31) / 32; i += kMoveBlock) s_flag_bits[i] = 0u;
        reinterpret_cast<uint4*>(s_owner)[2 * tid] = make_uint4(0u, 0u, 0u, 0u);
        reinterpret_cast<uint4*>(s_owner)[2 * tid + 1] = make_uint4(0u, 0u, 0u, 0u);
        __syncthreads();
        // the window's loads in batches of kWindowBatch per thread, each batch
        // in flight at once (one batch covers up to 2048 tiles)
        for (uint32_t i0 = 0; i0 < ntiles; i0 += kMoveBlock * kWindowBatch) {  // uniform
            uint32_t win[kWindowBatch];
#pragma unroll
            for (int u = 0; u < kWindowBatch; ++u) {
                const uint32_t i = i0 + tid + u * kMoveBlock;
                win[u] = i < ntiles ? a.tile_excl[t0 + i] : 0u;
            }
#pragma unroll
            for (int u = 0; u < kWindowBatch; ++u) {
                const uint32_t i = i0 + tid + u * kMoveBlock;
                if (i < ntiles) {
                    s_off[i] = win[u] & ~kOverflow;
                    if (win[u] & kOverflow) atomicOr(&s_flag_bits[i / 32], 1u << (i % 32));
                }
            }
        }
        __syncthreads();
        const uint64_t x0 = static_cast<uint64_t>(m) * span_items;
        const uint64_t x1 = x0 + span_items < total ? x0 + span_items : total;
        const uint32_t lo = pairs_before(x0, t0, s_off[0]);
        uint32_t hi = x1 == total ? static_cast<uint32_t>(k) : pairs_before(x1, t1, s_off[ntiles - 1]);
        // lo <= hi <= lo + span_items and hi <= k hold by construction; the
        // clamps only keep the accesses below inside their buffers
        hi = hi < lo ? lo : hi;
        hi = hi - lo <= span_items ? hi : lo + span_items;
        hi = static_cast<int64_t>(hi) <= k ? hi : static_cast<uint32_t>(k);
        hi = hi < lo ? lo : hi;
        // Tile q owns the positions from its offset up to the next tile's;
        // only the first tile of the window can start before lo.
        for (uint32_t q = tid; q < ntiles; q += kMoveBlock) {
            const uint32_t off = s_off[q];
            const bool owner = q + 1 == ntiles || s_off[q + 1] != off;
            if (owner && off < hi) s_owner[(off > lo ? off : lo) - lo] = static_cast<uint16_t>(q);
        }
        __syncthreads();
        block_max_scan(s_owner, tid, s_wave_max);
        for (uint32_t j0 = lo + tid; j0 < hi; j0 += kMoveBlock * kMoveBatch) {
            size_t src[kMoveBatch];
            bool live[kMoveBatch];
#pragma unroll
            for (int u = 0; u < kMoveBatch; ++u) {
                const uint32_t j = j0 + u * kMoveBlock;
                live[u] = j < hi;
                src[u] = 0;
                if (live[u]) {
                    const uint32_t q = s_owner[j - lo];
                    live[u] = !((s_flag_bits[q / 32] >> (q % 32)) & 1u);
                    src[u] = static_cast<size_t>(t0 + q) * kStageCap + (j - s_off[q]);
                }
            }
            // Loads outside any branch (a lane with nothing to copy reads
            // stage[0], inside the buffer since k > 0), then one wait for all
            // of them: the stores below, each under its own branch, would
            // otherwise wait for the vector-memory counter to drain, stores
            // included, before each other.
            uint2 pair[kMoveBatch];
#pragma unroll
            for (int u = 0; u < kMoveBatch; ++u) pair[u] = a.stage[src[u]];
            __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
#pragma unroll
            for (int u = 0; u < kMoveBatch; ++u) {
                if (live[u]) {
                    const uint32_t j = j0 + u * kMoveBlock;
                    a.out_idx[j] = static_cast<int32_t>(pair[u].x);
                    a.out_val[j] = __uint_as_float(pair[u].y);
                }
            }
        }
        __syncthreads();  // the window is reloaded for the next piece
    }
}

// Move kernel: a fixed grid walks the merged sequence of tiles and output
// pairs in pieces of move_span items (kMoveSpan, or a smaller size where the
// sequence is short: more, shorter pieces), so every piece costs about the same whatever the clustering of the
// selection: many pairs from few tiles, or few pairs scattered over many
// tiles.  Piece m's items lie in the tiles from split_tile[m] to
// split_tile[m + 1] (recorded by the scan kernel), at most move_span + 1 of
// them, and it holds the output positions [lo, hi).  The
// tiles' output offsets go to LDS; every tile that is the last of its offset
// (so the one that owns the positions from that offset on) writes its window
// index at its first position in the piece, and a running maximum fills in the
// owner of every position.  Each position then copies its staged pair with a
// coalesced write.  Before its pieces, every workgroup redoes its share of the
// flagged tiles, so a dense region of the partition costs the whole grid a
// second pass over it rather than one workgroup a serial one.
template <int VEC, bool SWEEP, bool HINT = false>
__device__ __forceinline__ void move_pieces(const LaunchArgs& a, const SweepTable* tbl) {
    constexpr int WAVES = kMoveBlock / kWaveSize;
    __shared__ double s_sq[WAVES];

    const int tid = threadIdx.x;
    const int lane = tid & (kWaveSize - 1);
    // The split words of this workgroup's first piece are read together with
    // the count (one round trip, not two); they are used only if the piece
    // exists, and then the scan kernel wrote them.  Both indices lie inside
    // the split array, which has room for the largest grid plus one.
    const uint32_t first_t0 = a.split_tile[blockIdx.x];
    const uint32_t first_t1 = a.split_tile[blockIdx.x + 1];
    // both counts in one load: the flagged-tile count must not wait for k
    const longlong2 counts = *reinterpret_cast<const longlong2*>(a.count_out);
    const int64_t k = counts.x;
    const uint32_t flagged = flagged_count(a, counts.y);
    // What goes to mapped host memory (the counts; in a sweep also each
    // segment's count and each chunk's squared norm) is stored by the grid's
    // last workgroups, which have the fewest pieces (none when the grid
    // exceeds the pieces), as early as they can: each such store is a bus
    // round trip, which then overlaps the other workgroups' moves instead of
    // following them.  (Measured: ResNet-50 rank 0 step 17.0-17.1 against
    // 17.4-17.5 us, ResNet-18 sweep 41.6-42.3 against 43.1-43.8 us.)
    const uint32_t host_wg = gridDim.x - 1;
    if (blockIdx.x == host_wg) {
        if (tid == 0) {  // the scan kernel has finished both counts
            a.host_count[0] = k;
            a.host_count[1] = flagged;
        }
        if constexpr (SWEEP) {
            // Each segment's count: the difference of the global offsets of
            // its first tile and of the next segment's first tile.
            if (tid < static_cast<int>(tbl->count)) {
                const uint32_t t0 = tbl->seg[tid].tile_first, t1 = tbl->seg[tid + 1].tile_first;
                const int64_t e0 = t0 < a.num_tiles ? (a.tile_excl[t0] & ~kOverflow) : k;
                const int64_t e1 = t1 < a.num_tiles ? (a.tile_excl[t1] & ~kOverflow) : k;
                a.host_count[2 + tid] = t1 > t0 ? e1 - e0 : 0;
            }
        }
    }
    if (k != 0) move_work<VEC, SWEEP, HINT>(a, tbl, k, flagged, first_t0, first_t1);
    if constexpr (SWEEP) {
        // Each chunk's squared norm, its tiles' norms added in a fixed order
        // (each thread its tiles in increasing order, then the workgroup sum);
        // the host adds a segment's chunks in increasing order.  The stream
        // workgroups stored the tile norms in an earlier launch, so they are
        // read here, not by the scan workgroups of a fused launch.
        for (uint32_t c = host_wg - blockIdx.x; c < a.num_chunks; c += gridDim.x) {  // uniform: from the grid's end
            uint32_t first, end;
            chunk_tiles<true>(a, tbl, c, first, end);
            double sq = 0.0;
            for (uint32_t t = first + tid; t < end; t += kMoveBlock) sq += a.tile_sumsq[t];
            const double total = block_sum<WAVES>(sq, lane, tid / kWaveSize, s_sq);
            if (tid == 0) a.host_sumsq[c] = total;
            __syncthreads();  // s_sq is written again for the next chunk
        }
    }
}

template <int VEC>
__global__ __launch_bounds__(kMoveBlock) void move_kernel(LaunchArgs a) {
    move_pieces<VEC, false>(a, nullptr);
}

// The move kernel after the hint kernels' stream pass: a flagged tile it redoes
// also sets only the residual of values at or above theta_zero to +0.
template <int VEC>
__global__ __launch_bounds__(kMoveBlock) void move_hint_kernel(LaunchArgs a) {
    move_pieces<VEC, false, true>(a, nullptr);
}

template <int VEC>
__global__ __launch_bounds__(kMoveBlock) void move_sweep_kernel(LaunchArgs a, SweepTable tbl) {
    move_pieces<VEC, true>(a, &tbl);
}

// ---------------------------------------------------------------------------
// Ticket schedule (variant 1)
// ---------------------------------------------------------------------------

constexpr int kTicketBlock = 256;

template <int VEC, int ROWS>
__global__ __launch_bounds__(kTicketBlock) void ticket_kernel(LaunchArgs a) {
    constexpr int WAVES = kTicketBlock / kWaveSize;
    static_assert(VEC * ROWS * kTicketBlock == kTicketTile, "tile size");
    __shared__ uint32_t s_tile;
    __shared__ uint32_t s_exclusive;
    __shared__ uint32_t s_wave_total[ROWS * WAVES];

    const int tid = threadIdx.x;
    const int lane = tid & (kWaveSize - 1);
    const int wave = tid / kWaveSize;

    if (tid == 0) s_tile = draw_ticket(a.ticket, a.num_tiles - 1);
    __syncthreads();
    const uint32_t tile = s_tile;
    if (tile >= a.num_tiles) return;  // only reachable if the counter was not rearmed

    Tile<VEC, ROWS, kTicketBlock> t;
    uint32_t lane_rank[ROWS], row_count[ROWS], row_base[ROWS];
    load_tile<VEC, ROWS, kTicketBlock, false>(a, a.base + static_cast<int64_t>(tile) * kTicketTile, tid, t);
    const uint32_t sel = compute_tile(a, tid, t);
    store_residual<VEC, ROWS, kTicketBlock, false>(a, tid, t, sel);
    wave_ranks<VEC, ROWS>(sel, lane_rank, row_count);
    const uint32_t count = tile_ranks<ROWS, WAVES>(row_count, lane, wave, s_wave_total, row_base);
    if (wave == 0) {
        const uint64_t tag = static_cast<uint64_t>(a.epoch) << kEpochShift;
        uint32_t excl = 0;
        if (tile == 0) {
            if (lane == 0) store_status(&a.status[0], tag | kFlagInclusive | count);
        } else {
            if (lane == 0) store_status(&a.status[tile], tag | kFlagAggregate | count);
            excl = lookback(a.status, tile, a.epoch, lane);
            if (lane == 0) store_status(&a.status[tile], tag | kFlagInclusive | (excl + count));
        }
        if (lane == 0) {
            s_exclusive = excl;
            if (tile == a.num_tiles - 1) {
                a.count_out[0] = static_cast<int64_t>(excl) + count;
                a.host_count[0] = static_cast<int64_t>(excl) + count;
                a.host_count[1] = 0;
            }
        }
    }
    __syncthreads();
    scatter_pairs(a, tid, t, sel, s_exclusive, row_base, lane_rank);
}

// ---------------------------------------------------------------------------
// Error-feedback accumulation outside the searched partition
// ---------------------------------------------------------------------------

// residual = grad + residual (one binary32 addition per value) over the tiles
// of two ranges, with the stream kernel's tile shape and non-temporal
// accesses; every value is written back, nothing is selected.
template <int VEC, int ROWS>
__global__ __launch_bounds__(kStreamBlock) void accumulate_kernel(AccumulateArgs acc) {
    static_assert(VEC * ROWS * kStreamBlock == kStreamTile, "tile size");
    uint32_t tile = blockIdx.x;
    int r = 0;
    if (tile >= acc.tiles[0]) {
        tile -= acc.tiles[0];
        r = 1;
    }
    LaunchArgs a{};
    a.grad = acc.grad;
    a.residual = acc.residual;
    a.start = acc.start[r];
    a.end = acc.end[r];
    const int tid = threadIdx.x;
    Tile<VEC, ROWS, kStreamBlock> t;
    load_tile<VEC, ROWS, kStreamBlock, true>(a, acc.base[r] + static_cast<int64_t>(tile) * kStreamTile, tid, t);
#pragma unroll
    for (int row = 0; row < ROWS; ++row)
#pragma unroll
        for (int c = 0; c < VEC; ++c) t.v[row][c] = t.v[row][c] + t.e[row][c];
    store_residual<VEC, ROWS, kStreamBlock, true>(a, tid, t, 0u);
}

// Refuses a launch whose kernels would dereference a null scratch or output
// pointer: every address a schedule's kernels use must be set by the host.
template <class... P>
bool all_set(const P*... p) {
    return ((p != nullptr) && ...);
}

bool staged_args_set(const LaunchArgs& a) {
    return all_set(a.grad, a.residual, a.out_idx, a.out_val, a.count_out, a.host_count, a.tile_excl, a.flagged_list,
                   a.split_tile, a.stage, a.chunk_status);
}

}  // namespace

hipError_t launch_accumulate(const AccumulateArgs& args, bool vec4, hipStream_t stream) {
    const uint32_t blocks = args.tiles[0] + args.tiles[1];
    if (blocks == 0) return hipSuccess;
    if (vec4)
        hipLaunchKernelGGL((accumulate_kernel<4, 1>), dim3(blocks), dim3(kStreamBlock), 0, stream, args);
    else
        hipLaunchKernelGGL((accumulate_kernel<1, 4>), dim3(blocks), dim3(kStreamBlock), 0, stream, args);
    return hipGetLastError();
}

int64_t tile_base_for(const float* grad, int64_t start, bool vec4) {
    if (!vec4) return start;
    const uintptr_t addr = reinterpret_cast<uintptr_t>(grad + start);
    return start - static_cast<int64_t>((addr & 15u) / sizeof(float));
}

hipError_t launch_staged(const LaunchArgs& args, bool vec4, hipStream_t stream) {
    if (!staged_args_set(args) || !args.tile_counts) return hipErrorInvalidValue;
    const dim3 grid_stream(args.num_tiles), grid_scan(args.num_chunks), grid_move(args.move_blocks);
    const dim3 bs(kStreamBlock);
    const bool hint = args.theta_zero > args.theta_f;
    if (vec4) {
        if (hint) {
            hipLaunchKernelGGL((stream_hint_kernel<4, 1>), grid_stream, bs, 0, stream, args);
            hipLaunchKernelGGL(scan_kernel, grid_scan, dim3(kScanBlock), 0, stream, args);
            hipLaunchKernelGGL(move_hint_kernel<4>, grid_move, dim3(kMoveBlock), 0, stream, args);
            return hipGetLastError();
        }
        hipLaunchKernelGGL((stream_kernel<4, 1>), grid_stream, bs, 0, stream, args);
        hipLaunchKernelGGL(scan_kernel, grid_scan, dim3(kScanBlock), 0, stream, args);
        hipLaunchKernelGGL(move_kernel<4>, grid_move, dim3(kMoveBlock), 0, stream, args);
    } else {
        if (hint) {
            hipLaunchKernelGGL((stream_hint_kernel<1, 4>), grid_stream, bs, 0, stream, args);
            hipLaunchKernelGGL(scan_kernel, grid_scan, dim3(kScanBlock), 0, stream, args);
            hipLaunchKernelGGL(move_hint_kernel<1>, grid_move, dim3(kMoveBlock), 0, stream, args);
            return hipGetLastError();
        }
        hipLaunchKernelGGL((stream_kernel<1, 4>), grid_stream, bs, 0, stream, args);
        hipLaunchKernelGGL(scan_kernel, grid_scan, dim3(kScanBlock), 0, stream, args);
        hipLaunchKernelGGL(move_kernel<1>, grid_move, dim3(kMoveBlock), 0, stream, args);
    }
    return hipGetLastError();
}

hipError_t launch_fused(const LaunchArgs& args, bool vec4, hipStream_t stream) {
    if (!staged_args_set(args) || !args.tile_words) return hipErrorInvalidValue;
    const dim3 grid_fused(args.num_tiles + args.num_chunks), grid_move(args.move_blocks);
    const bool hint = args.theta_zero > args.theta_f;
    if (vec4) {
        if (hint) {
            hipLaunchKernelGGL((stream_scan_hint_kernel<4, 1>), grid_fused, dim3(kStreamBlock), 0, stream, args);
            hipLaunchKernelGGL(move_hint_kernel<4>, grid_move, dim3(kMoveBlock), 0, stream, args);
            return hipGetLastError();
        }
        hipLaunchKernelGGL((stream_scan_kernel<4, 1>), grid_fused, dim3(kStreamBlock), 0, stream, args);
        hipLaunchKernelGGL(move_kernel<4>, grid_move, dim3(kMoveBlock), 0, stream, args);
    } else {
        if (hint) {
            hipLaunchKernelGGL((stream_scan_hint_kernel<1, 4>), grid_fused, dim3(kStreamBlock), 0, stream, args);
            hipLaunchKernelGGL(move_hint_kernel<1>, grid_move, dim3(kMoveBlock), 0, stream, args);
            return hipGetLastError();
        }
        hipLaunchKernelGGL((stream_scan_kernel<1, 4>), grid_fused, dim3(kStreamBlock), 0, stream, args);
        hipLaunchKernelGGL(move_kernel<1>, grid_move, dim3(kMoveBlock), 0, stream, args);
    }
    return hipGetLastError();
}

hipError_t launch_sweep(const LaunchArgs& args, const SweepTable& table, bool vec4, bool fused, hipStream_t stream) {
    if (!staged_args_set(args) || !all_set(args.tile_sumsq, args.host_sumsq) ||
        !(fused ? args.tile_words != nullptr : args.tile_counts != nullptr))
        return hipErrorInvalidValue;
    const dim3 grid_stream(args.num_tiles), grid_scan(args.num_chunks), grid_move(args.move_blocks);
    const dim3 bs(kStreamBlock);
    if (fused) {
        const dim3 grid_fused(args.num_tiles + args.num_chunks);
        if (vec4) {
            hipLaunchKernelGGL((stream_scan_sweep_kernel<4, 1>), grid_fused, bs, 0, stream, args, table);
            hipLaunchKernelGGL(move_sweep_kernel<4>, grid_move, dim3(kMoveBlock), 0, stream, args, table);
        } else {
            hipLaunchKernelGGL((stream_scan_sweep_kernel<1, 4>), grid_fused, bs, 0, stream, args, table);
            hipLaunchKernelGGL(move_sweep_kernel<1>, grid_move, dim3(kMoveBlock), 0, stream, args, table);
        }
        return hipGetLastError();
    }
    if (vec4) {
        hipLaunchKernelGGL((stream_sweep_kernel<4, 1>), grid_stream, bs, 0, stream, args, table);
        hipLaunchKernelGGL(scan_sweep_kernel, grid_scan, dim3(kScanBlock), 0, stream, args, table);
        hipLaunchKernelGGL(move_sweep_kernel<4>, grid_move, dim3(kMoveBlock), 0, stream, args, table);
    } else {
        hipLaunchKernelGGL((stream_sweep_kernel<1, 4>), grid_stream, bs, 0, stream, args, table);
        hipLaunchKernelGGL(scan_sweep_kernel, grid_scan, dim3(kScanBlock), 0, stream, args, table);
        hipLaunchKernelGGL(move_sweep_kernel<1>, grid_move, dim3(kMoveBlock), 0, stream, args, table);
    }
    return hipGetLastError();
}

hipError_t launch_ticket(const LaunchArgs& args, bool vec4, hipStream_t stream) {
    if (!all_set(args.grad, args.residual, args.out_idx, args.out_val, args.count_out, args.host_count, args.status,
                 args.ticket))
        return hipErrorInvalidValue;
    const dim3 grid(args.num_tiles), block(kTicketBlock);
    if (vec4)
        hipLaunchKernelGGL((ticket_kernel<4, 4>), grid, block, 0, stream, args);
    else
        hipLaunchKernelGGL((ticket_kernel<1, 16>), grid, block, 0, stream, args);
    return hipGetLastError();
}

}  // namespace micro
