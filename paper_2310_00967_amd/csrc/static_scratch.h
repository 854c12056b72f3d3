// Internal interface of the allocation-free step's device scratch
// (static_scratch.hip).  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sparsify_kernel.h"

namespace micro {

// The allocation-free step runs the one-pass ticket schedule with its
// scratch in one static device array per device, of kStaticScratchWords
// 64-bit words (4 MiB + 256 bytes):
//   word 0                    the ticket counter (0 between launches)
//   words 1, 2                count_out: the selected count, the flagged word
//   words 3, 4                where the kernel stores the counts it would
//                             otherwise store into mapped host memory
//   words kStaticHeaderWords  one look-back status word per tile, for up to
//   ...                       kStaticMaxTiles 4096-value tiles: a partition of
//                             up to 2^31 - 1 values (the int32 index range)
//                             plus the 16-byte alignment of its first tile
constexpr int64_t kStaticHeaderWords = 32;  // 256 bytes: the status words stay 256-byte aligned
constexpr int64_t kStaticMaxTiles = ((int64_t(1) << 31) + 2 + kTicketTile - 1) / kTicketTile;
constexpr int64_t kStaticScratchWords = kStaticHeaderWords + kStaticMaxTiles;

// The device address of the static scratch on the current device, looked up
// once per device with hipGetSymbolAddress and kept.  Thread-safe.
hipError_t static_scratch_current_device(uint64_t** words);

// words[0, n) = 0 with a fill kernel on `stream` (no memset node, so the
// clear is also valid inside a captured graph).
hipError_t launch_clear_words(uint64_t* words, int64_t n, hipStream_t stream);

}  // namespace micro
