// Internal interface between the host library and the gfx950 kernels of the
// sparsify step.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace micro {

// Staged schedule: values per stream tile (one 256-thread workgroup), staged
// pairs per tile, tiles per scan chunk (one 256-thread workgroup), items per
// move piece.  The move kernel walks the merged sequence of tiles and output
// pairs (each tile is one item, followed by one item per selected value of
// the tile) in pieces of move_span items (kMoveSpan, or kMoveSpanSmall / kMoveSpanTiny for a
// short sequence), so a piece holds at most kMoveSpan pairs and touches at
// most kMoveSpan + 1 tiles.
constexpr int kStreamTile = 1024;
constexpr int kStreamBlock = 256;
constexpr uint32_t kStageCap = 256;
constexpr int kChunkTiles = 1024;
constexpr int kScanBlock = 256;
constexpr int kMoveSpan = 4096;        // largest move piece (LDS arrays are sized for it)
constexpr int kMoveSpanSmall = 1024;   // move piece of a short merged sequence
constexpr int kMoveSpanTiny = 512;     // move piece of a very short one
constexpr int kMoveBlock = 256;
constexpr uint32_t kMoveGrid = 2048;  // largest move grid (eight workgroups per compute unit)
static_assert((kMoveSpan & (kMoveSpan - 1)) == 0 && (kMoveSpanSmall & (kMoveSpanSmall - 1)) == 0 &&
                  (kMoveSpanTiny & (kMoveSpanTiny - 1)) == 0 && kMoveSpanTiny <= kMoveSpanSmall,
              "piece sizes are powers of two: the kernels divide by them with shifts");
// Ticket schedule: values per tile (256 threads, four dwordx4 per lane).
constexpr int kTicketTile = 4096;

// Fused stream-and-scan launch: num_tiles + num_chunks workgroups.  The scan
// workgroup of chunk c follows the stream workgroup of the last tile of chunk
// c + kChunkLag, so it is dispatched when its own chunk's tiles have had about
// kChunkLag * kChunkTiles dispatches to finish and scans while the stream goes
// on; the chunks that have no such tile (the last kChunkLag or so) follow all
// tiles, in order.  Every scan workgroup therefore comes after its chunk's
// tiles and after the scan workgroups of all lower chunks.
constexpr uint32_t kChunkLag = 2;

struct FusedRole {
    bool scan;      // a scan workgroup (else a stream workgroup)
    uint32_t item;  // its chunk, or its tile
};

// Role of workgroup b of the fused launch.  Chunk c (num_chunks of them)
// sits at position min(num_tiles, (c + kChunkLag + 1) * kChunkTiles) + c.
// Chunks c < c0 = max(0, floor(num_tiles / kChunkTiles) - kChunkLag) are the
// interleaved ones, at (c + kChunkLag + 1) * (kChunkTiles + 1) - (kChunkLag + 1);
// the others sit at num_tiles + c.
__host__ __device__ inline FusedRole fused_role(uint32_t b, uint32_t num_tiles, uint32_t num_chunks) {
    const uint32_t whole = num_tiles / kChunkTiles;
    const uint32_t c0 = whole > kChunkLag ? whole - kChunkLag : 0u;
    if (b >= num_tiles + c0) return {true, b - num_tiles};
    const uint32_t q = b + kChunkLag + 1;
    const uint32_t g = q / (kChunkTiles + 1);
    if (q % (kChunkTiles + 1) == 0 && g >= kChunkLag + 1) return {true, g - kChunkLag - 1};
    const uint32_t before = g > kChunkLag ? (g - kChunkLag < c0 ? g - kChunkLag : c0) : 0u;
    (void)num_chunks;
    return {false, b - before};
}

// Bits of a look-back status word (one 64-bit word per tile or chunk):
//   [0, 32)  count: the item's own selected count (aggregate) or the
//            inclusive prefix of selected counts through this item
//   [32, 34) flag: 1 = aggregate published, 2 = inclusive prefix published
//   [34, 64) epoch of the launch that wrote it; words of older launches
//            read as "not yet published", so the arrays are never cleared
//            between launches
constexpr int kEpochShift = 34;
constexpr uint32_t kMaxEpoch = (1u << 30) - 1;

// Sweep of every partition of one vector with one launch of each staged
// kernel: the partitions are segments of the tile sequence (each with its own
// threshold, range and tile grid), and scan chunks never straddle two of them.
// The pairs of all segments form one compaction in index order.
constexpr int kMaxSweep = 64;

struct SweepSegment {
    int64_t start;          // partition [start, end)
    int64_t end;
    int64_t base;           // global index of the segment's first tile's first value
    float theta_f;          // the segment's binary32 threshold
    uint32_t tile_first;    // first global tile of the segment
    uint32_t chunk_first;   // first global scan chunk of the segment
    uint32_t wg_first;      // fused sweep: first workgroup of the segment (its tiles and chunks, laid
                            // out by fused_role); seg[count].wg_first = the launch's workgroups
};

struct SweepTable {
    uint32_t count;                       // segments
    uint32_t pad;
    SweepSegment seg[kMaxSweep + 1];      // seg[count]: tile_first / chunk_first = the totals
};

struct LaunchArgs {
    const float* grad;      // device, global indexing
    float* residual;        // device, global indexing
    int32_t* out_idx;       // device, P entries
    float* out_val;         // device, P entries
    int64_t start;          // partition [start, end)
    int64_t end;
    int64_t base;           // global index of tile 0's first value (<= start)
    float theta_f;          // smallest binary32 >= theta
    uint32_t epoch;         // 1 .. kMaxEpoch
    uint32_t num_tiles;     // tiles covering [base, end)
    int64_t* count_out;     // device: [0] selected count, [1] (epoch << 32) | flagged tiles (redone by the
                            // move kernel; a word of an older launch counts none)
    int64_t* host_count;    // mapped pinned host memory: the final count_out, stored by the last kernel;
                            // a sweep adds each segment's count from [2] on
    // staged schedule
    uint32_t* tile_counts;  // num_tiles counts (bit 31: tile left to the scan kernel)
    uint64_t* tile_words;   // fused schedule: num_tiles epoch-tagged counts (status word layout)
    uint32_t* tile_excl;    // num_tiles output offsets (bit 31: flagged tile)
    uint32_t* flagged_list; // count_out[1] flagged tiles, in no particular order
    uint32_t* split_tile;   // >= ceil((num_tiles + P) / kMoveSpan) tiles holding each piece's first item
    double* tile_sumsq;     // sweep: per tile, squared norm of its new residual (binary64)
    double* host_sumsq;     // sweep: mapped host memory, per scan chunk the sum of its tiles'
                            // squared norms (the host adds each segment's chunks in order)
    uint32_t move_blocks;   // workgroups of the move kernel
    uint32_t move_span;     // items per move piece: kMoveSpan, kMoveSpanSmall or kMoveSpanTiny (a power of two)
    uint2* stage;           // num_tiles * kStageCap staged (index, value bits) pairs
    uint32_t num_chunks;    // ceil(num_tiles / kChunkTiles)
    uint64_t* chunk_status;             // >= num_chunks look-back words
    // ticket schedule
    uint64_t* status;                   // >= num_tiles look-back words
    unsigned long long* ticket;         // 0 at launch, rearmed by the kernel
    // staged schedule, theta_zero > theta_f: of the selected values only those
    // with |acc| >= theta_zero have their residual set to +0; the others keep
    // acc there (the top-k comparator's step at a hint's bound)
    float theta_zero;
};

// Error-feedback accumulation outside the searched partition (Algorithm 1,
// every element accumulates its new gradient): residual = grad + residual
// over ranges [start[r], end[r]), r = 0, 1, in tiles of kStreamTile values
// whose first tile starts at base[r] (<= start[r]); workgroups
// [0, tiles[0]) take range 0, the next tiles[1] range 1.
struct AccumulateArgs {
    const float* grad;
    float* residual;
    int64_t start[2];
    int64_t end[2];
    int64_t base[2];
    uint32_t tiles[2];
};

// Global index of tile 0's first value: the start rounded down so that
// grad + base is 16-byte aligned (vectorised kernels), or the start.
int64_t tile_base_for(const float* grad, int64_t start, bool vec4);

// vec4: grad and residual share their 16-byte phase (dwordx4 kernels), else
// the scalar-load kernels.  Each returns the launch status.  launch_staged and
// launch_fused take the kernels that honour theta_zero when it is above
// theta_f.
hipError_t launch_staged(const LaunchArgs& args, bool vec4, hipStream_t stream);
// The staged schedule with its stream and scan kernels fused into one launch
// (num_tiles + num_chunks workgroups, roles from fused_role).  Its waits end
// because every chunk workgroup waits only for workgroups of lower index in
// the same launch and each XCD dispatches its workgroups in index order.
hipError_t launch_fused(const LaunchArgs& args, bool vec4, hipStream_t stream);
hipError_t launch_ticket(const LaunchArgs& args, bool vec4, hipStream_t stream);
// The sweep: num_tiles / num_chunks are the totals over the table's segments.
// fused: the stream and scan passes in one launch of num_tiles + num_chunks
// workgroups, each segment's workgroups from its wg_first on as fused_role
// lays out a single partition's.
hipError_t launch_sweep(const LaunchArgs& args, const SweepTable& table, bool vec4, bool fused, hipStream_t stream);
hipError_t launch_accumulate(const AccumulateArgs& args, bool vec4, hipStream_t stream);

// Union kernels (union_kernel.hip).  Gather and reset at the union of the
// workers' selections: out[q] = own_val[q - own_first] for q in
// [own_first, own_first + own_count), else out[q] = residual[idx[q]] and
// residual[idx[q]] = +0 (indices outside [0, n): no access, out[q] = NaN).
hipError_t launch_union_gather(float* residual, int64_t n, const int32_t* idx, int64_t m, int64_t own_first,
                               int64_t own_count, const float* own_val, float* out, hipStream_t stream);
// Model update: x[idx[q]] = x[idx[q]] - sums[q] / world, q in [0, m)
// (indices outside [0, n_x) skipped).
hipError_t launch_sparse_update(float* x, int64_t n_x, const int32_t* idx, const float* sums, int64_t m,
                                float world, hipStream_t stream);

}  // namespace micro
