// Internal interface between the host library and the gfx950 kernels of the
// sparsify step.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace micro {

// Elements per tile; the same for every kernel variant so one status array
// sized for the largest partition serves all of them.
constexpr int kTileElems = 4096;

// Bits of a tile status word (one 64-bit word per tile):
//   [0, 32)  count: the tile's own selected count (aggregate) or the
//            inclusive prefix of selected counts through this tile
//   [32, 34) flag: 1 = aggregate published, 2 = inclusive prefix published
//   [34, 64) epoch of the launch that wrote it; words of older launches
//            read as "not yet published", so the array is never cleared
//            between launches
constexpr int kEpochShift = 34;
constexpr uint32_t kMaxEpoch = (1u << 30) - 1;

struct LaunchArgs {
    const float* grad;      // device, global indexing
    float* residual;        // device, global indexing
    int32_t* out_idx;       // device, P entries
    float* out_val;         // device, P entries
    int64_t start;          // partition [start, end)
    int64_t end;
    int64_t base;           // global index of tile 0's first element (<= start)
    float theta_f;          // smallest binary32 >= theta
    uint64_t* status;       // device, >= num_tiles words
    unsigned long long* ticket;  // device tile ticket counter: 0 at launch,
                                 // reset to 0 by the workgroup that draws the
                                 // last ticket
    uint32_t epoch;         // 1 .. kMaxEpoch
    uint32_t num_tiles;
    int64_t* count_out;     // device word: receives the selected count
};

// Chooses the vectorised (dwordx4) kernel when grad and residual share their
// 16-byte phase, else the scalar-load kernel; `base` must be set accordingly
// (see tile_base_for).  Returns the launch status.
hipError_t launch_sparsify(const LaunchArgs& args, bool vec4, hipStream_t stream);

// Global index of tile 0's first element: the start rounded down so that
// grad + base is 16-byte aligned (vectorised kernel), or the start itself.
int64_t tile_base_for(const float* grad, int64_t start, bool vec4);

}  // namespace micro
