// gfx950 kernel of MiCRO's per-worker sparsify step (arXiv 2310.00967).
//
// One launch streams a worker's partition [start, end) once (Sec. 4.1,
// Sec. 4.2): every workgroup takes the next tile by ticket, reads grad and
// residual (dwordx4 per lane), forms acc = grad + residual (Sec. 2, error
// feedback), tests |acc| >= theta_f, writes residual = selected ? +0 : acc
// (Algorithm 1, reset and carry of the local error) and compacts the selected
// (index, acc) pairs in index order (Algorithm 1, selection and gathering).
//
// Order-preserving compaction, all in one pass:
//   * per wavefront row: one ballot per element slot and mbcnt give each
//     lane's rank among the selected elements before it in the row;
//   * per workgroup: the wavefront row totals go through LDS, giving each
//     row's offset inside the tile and the tile's count;
//   * across workgroups: decoupled look-back over one 64-bit status word per
//     tile (count | flag | epoch).  Wavefront 0 inspects 64 predecessors per
//     round with agent-scope atomic loads, so a tile rarely waits longer than
//     one round trip through the coherent memory level shared by all XCDs.
// Tiles are claimed in increasing order through a ticket counter, so a tile
// only ever waits for tiles claimed earlier by workgroups that are already
// running: the look-back always makes progress.
#include "sparsify_kernel.h"

namespace micro {
namespace {

constexpr int kBlock = 256;
constexpr int kWaveSize = 64;
constexpr int kWaves = kBlock / kWaveSize;

constexpr uint64_t kCountMask = 0xffffffffull;
constexpr uint64_t kFlagAggregate = 1ull << 32;
constexpr uint64_t kFlagInclusive = 2ull << 32;
constexpr uint64_t kFlagMask = 3ull << 32;

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWaveSize);
    return v;
}

__device__ __forceinline__ uint64_t load_status(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void store_status(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Executed by all 64 lanes of one wavefront.  Publishes the tile's aggregate,
// sums predecessors back to the nearest inclusive prefix, publishes the
// tile's inclusive prefix and returns the exclusive prefix (uniform).
// The count and its flag share one 64-bit word, so relaxed atomics suffice:
// a reader either sees the whole published word or an older one.
__device__ uint32_t decoupled_lookback(uint64_t* status, uint32_t tile, uint32_t epoch,
                                       uint32_t tile_count, int lane) {
    const uint64_t tag = static_cast<uint64_t>(epoch) << kEpochShift;
    if (tile == 0) {
        if (lane == 0) store_status(&status[0], tag | kFlagInclusive | tile_count);
        return 0;
    }
    if (lane == 0) store_status(&status[tile], tag | kFlagAggregate | tile_count);

    uint32_t exclusive = 0;
    int64_t top = static_cast<int64_t>(tile) - 1;
    for (;;) {
        const int64_t p = top - lane;
        // Positions before tile 0 read as an inclusive prefix of zero; tile 0
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
        if (inc_mask) break;
        top -= kWaveSize;
    }
    if (lane == 0) store_status(&status[tile], tag | kFlagInclusive | (exclusive + tile_count));
    return exclusive;
}

// VEC consecutive elements per lane per row, ROWS rows per tile; element
// (row, thread, c) of a tile sits at tile_base + (row * kBlock + thread) * VEC + c,
// which is also its order in the compacted output.
template <int VEC, int ROWS>
__global__ __launch_bounds__(kBlock) void sparsify_kernel(LaunchArgs a) {
    static_assert(VEC * ROWS * kBlock == kTileElems, "tile size");
    __shared__ uint32_t s_tile;
    __shared__ uint32_t s_exclusive;
    __shared__ uint32_t s_wave_total[ROWS * kWaves];

    const int tid = threadIdx.x;
    const int lane = tid & (kWaveSize - 1);
    const int wave = tid / kWaveSize;

    if (tid == 0) {
        const uint32_t t = static_cast<uint32_t>(atomicAdd(a.ticket, 1ull));
        // Every other workgroup of this launch has drawn its ticket before the
        // last one is drawn, so the counter can be rearmed for the next launch.
        if (t == a.num_tiles - 1) __hip_atomic_store(a.ticket, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_tile = t;
    }
    __syncthreads();
    const uint32_t tile = s_tile;
    if (tile >= a.num_tiles) return;  // only reachable if the counter was not rearmed
    const int64_t tile_base = a.base + static_cast<int64_t>(tile) * kTileElems;
    const bool interior = tile_base >= a.start && tile_base + kTileElems <= a.end;

    float acc[ROWS][VEC];
    bool sel[ROWS][VEC];

    if (interior) {
        // All loads of the tile are issued before any residual store, so each
        // lane keeps 2 * ROWS * VEC * 4 bytes in flight.
        if constexpr (VEC == 4) {
            f32x4 g[ROWS], e[ROWS];
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                const int64_t i = tile_base + static_cast<int64_t>(r * kBlock + tid) * VEC;
                g[r] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(a.grad + i));
            }
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                const int64_t i = tile_base + static_cast<int64_t>(r * kBlock + tid) * VEC;
                e[r] = *reinterpret_cast<const f32x4*>(a.residual + i);
            }
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
                const int64_t i = tile_base + static_cast<int64_t>(r * kBlock + tid) * VEC;
                f32x4 out;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    acc[r][c] = g[r][c] + e[r][c];
                    sel[r][c] = __builtin_fabsf(acc[r][c]) >= a.theta_f;
                    out[c] = sel[r][c] ? 0.0f : acc[r][c];
                }
                *reinterpret_cast<f32x4*>(a.residual + i) = out;
            }
        } else {
            float g[ROWS][VEC], e[ROWS][VEC];
#pragma unroll
            for (int r = 0; r < ROWS; ++r)
#pragma unroll
                for (int c = 0; c < VEC; ++c)
                    g[r][c] = __builtin_nontemporal_load(
                        a.grad + tile_base + static_cast<int64_t>(r * kBlock + tid) * VEC + c);
#pragma unroll
            for (int r = 0; r < ROWS; ++r)
#pragma unroll
                for (int c = 0; c < VEC; ++c)
                    e[r][c] = a.residual[tile_base + static_cast<int64_t>(r * kBlock + tid) * VEC + c];
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
#pragma unroll
                for (int c = 0; c < VEC; ++c) {
                    const int64_t i = tile_base + static_cast<int64_t>(r * kBlock + tid) * VEC + c;
                    acc[r][c] = g[r][c] + e[r][c];
                    sel[r][c] = __builtin_fabsf(acc[r][c]) >= a.theta_f;
                    a.residual[i] = sel[r][c] ? 0.0f : acc[r][c];
                }
            }
        }
    } else {
        // First or last tile of the partition: per-element guards.
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
#pragma unroll
            for (int c = 0; c < VEC; ++c) {
                const int64_t i = tile_base + static_cast<int64_t>(r * kBlock + tid) * VEC + c;
                const bool inside = i >= a.start && i < a.end;
                acc[r][c] = 0.0f;
                sel[r][c] = false;
                if (inside) {
                    acc[r][c] = a.grad[i] + a.residual[i];
                    sel[r][c] = __builtin_fabsf(acc[r][c]) >= a.theta_f;
                    a.residual[i] = sel[r][c] ? 0.0f : acc[r][c];
                }
            }
        }
    }

    // Rank of each lane's first selected element inside its wavefront row,
    // and the row totals of every wavefront.
    uint32_t lane_rank[ROWS];
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        uint32_t below = 0, total = 0;
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            const uint64_t m = __ballot(sel[r][c]);
            below += lanes_below(m);
            total += static_cast<uint32_t>(__popcll(m));
        }
        lane_rank[r] = below;
        if (lane == 0) s_wave_total[r * kWaves + wave] = total;
    }
    __syncthreads();

    uint32_t row_offset[ROWS];
    uint32_t running = 0;
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const uint32_t v = s_wave_total[r * kWaves + w];
            if (w == wave) row_offset[r] = running;
            running += v;
        }
    }
    const uint32_t tile_count = running;

    if (wave == 0) {
        const uint32_t excl = decoupled_lookback(a.status, tile, a.epoch, tile_count, lane);
        if (lane == 0) {
            s_exclusive = excl;
            if (tile == a.num_tiles - 1) *a.count_out = static_cast<int64_t>(excl) + tile_count;
        }
    }
    __syncthreads();
    const uint32_t exclusive = s_exclusive;

#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        uint32_t pos = exclusive + row_offset[r] + lane_rank[r];
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            if (sel[r][c]) {
                const int64_t i = tile_base + static_cast<int64_t>(r * kBlock + tid) * VEC + c;
                a.out_idx[pos] = static_cast<int32_t>(i);
                a.out_val[pos] = acc[r][c];
                ++pos;
            }
        }
    }
}

}  // namespace

int64_t tile_base_for(const float* grad, int64_t start, bool vec4) {
    if (!vec4) return start;
    const uintptr_t addr = reinterpret_cast<uintptr_t>(grad + start);
    return start - static_cast<int64_t>((addr & 15u) / sizeof(float));
}

hipError_t launch_sparsify(const LaunchArgs& args, bool vec4, hipStream_t stream) {
    const dim3 grid(args.num_tiles), block(kBlock);
    if (vec4)
        hipLaunchKernelGGL((sparsify_kernel<4, 4>), grid, block, 0, stream, args);
    else
        hipLaunchKernelGGL((sparsify_kernel<1, 16>), grid, block, 0, stream, args);
    return hipGetLastError();
}

}  // namespace micro
