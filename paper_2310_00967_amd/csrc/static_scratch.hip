// Device scratch of the allocation-free sparsify step: one static array in
// the code object, so every device the library runs on holds its own copy
// from the first launch until the process ends, and no call allocates.
//
// In host code the array's name only stands for the variable: its device
// address on each device comes from hipGetSymbolAddress, looked up once per
// device with that device current and kept; kernels receive that address.
#include "static_scratch.h"

#include <mutex>

// Zero when the code object is loaded on a device; see static_scratch.h for
// the layout.
static __device__ __align__(256) uint64_t scratch[micro::kStaticScratchWords];

namespace micro {
namespace {

constexpr int kMaxDevices = 64;
constexpr int kClearBlock = 256;

std::mutex g_lookup_mutex;
uint64_t* g_words[kMaxDevices] = {};

__global__ __launch_bounds__(kClearBlock) void clear_words_kernel(uint64_t* words, int64_t n) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kClearBlock + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * kClearBlock)
        words[i] = 0;
}

}  // namespace

hipError_t static_scratch_current_device(uint64_t** words) {
    int device = -1;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return e;
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_lookup_mutex);
    if (!g_words[device]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_words[device] = static_cast<uint64_t*>(p);
    }
    *words = g_words[device];
    return hipSuccess;
}

hipError_t launch_clear_words(uint64_t* words, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    int64_t blocks = (n + kClearBlock - 1) / kClearBlock;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(clear_words_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kClearBlock), 0, stream,
                       words, n);
    return hipGetLastError();
}

}  // namespace micro
