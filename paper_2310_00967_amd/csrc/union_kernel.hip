// gfx950 kernels around the exchange of MiCRO's Algorithm 1 (arXiv
// 2310.00967), on one worker's device:
//   union_gather_kernel  the accumulated values at the union of all workers'
//                        selected indices (the worker's contribution to the
//                        all-reduce), and their reset in the local error;
//   sparse_update_kernel the model update with the all-reduced sums averaged
//                        over the n workers.
// Both are bound by scattered-sector traffic and latency: one thread per
// union entry, contiguous index / value streams, monotone (sorted) gathers and
// scatters.
#include "sparsify_kernel.h"

namespace micro {
namespace {

constexpr int kUnionBlock = 256;

// Independent union entries per thread.  The gathers and scatters hit
// scattered 32-byte sectors, and the kernels are bound by how many such
// requests the memory system keeps in flight, not by instruction issue.  On a
// 3.35M-entry union, one entry per thread ran 5-7% faster than four (eight or
// sixteen were slower still), and 128- or 512-thread workgroups changed
// nothing.  The contiguous streams (the union indices, the sums, the outputs)
// and the scattered stores are non-temporal, since nothing here reads them
// again; that took another 3-5% off both kernels.  The scattered reads stay
// ordinary loads: non-temporal ones were 25% slower.  The gather's reset store
// follows its read at once instead of the output store that waits for the
// read's value (81.2 against 77.5-79.4 us on that union).
constexpr int kUnionPerThread = 1;

// The worker's own selection occupies union positions [own_first,
// own_first + own_count): those values are the step's outputs and their local
// error is already +0.  Every other position reads the accumulated value,
// which the error-feedback pass left in the residual, and resets it.  An index
// outside [0, n) touches nothing and yields a NaN.
__global__ __launch_bounds__(kUnionBlock) void union_gather_kernel(float* residual, int64_t n, const int32_t* idx,
                                                                   int64_t m, int64_t own_first, int64_t own_count,
                                                                   const float* own_val, float* out) {
    const int64_t first = (static_cast<int64_t>(blockIdx.x) * kUnionPerThread) * kUnionBlock + threadIdx.x;
    float v[kUnionPerThread];
    int32_t j[kUnionPerThread];
    bool own[kUnionPerThread];
#pragma unroll
    for (int u = 0; u < kUnionPerThread; ++u) {
        const int64_t q = first + static_cast<int64_t>(u) * kUnionBlock;
        own[u] = static_cast<uint64_t>(q - own_first) < static_cast<uint64_t>(own_count);
        j[u] = q < m && !own[u] ? __builtin_nontemporal_load(idx + q) : -1;
        if (j[u] >= n) j[u] = -2;  // out of range: no access
    }
#pragma unroll
    for (int u = 0; u < kUnionPerThread; ++u) {
        const int64_t q = first + static_cast<int64_t>(u) * kUnionBlock;
        v[u] = own[u] ? own_val[q - own_first] : (j[u] >= 0 ? residual[j[u]] : __builtin_nanf(""));
        // the reset goes out right behind the read of the same value (one
        // thread's accesses to one address are performed in order), without
        // waiting for the value to come back
        if (j[u] >= 0) __builtin_nontemporal_store(0.0f, residual + j[u]);
    }
#pragma unroll
    for (int u = 0; u < kUnionPerThread; ++u) {
        const int64_t q = first + static_cast<int64_t>(u) * kUnionBlock;
        if (q < m) __builtin_nontemporal_store(v[u], out + q);
    }
}

// x[idx[q]] = x[idx[q]] - sums[q] / n: one correctly rounded binary32
// division and one subtraction.  The indices are distinct, so no two threads
// touch one value; an index outside [0, n_x) is skipped.
__global__ __launch_bounds__(kUnionBlock) void sparse_update_kernel(float* x, int64_t n_x, const int32_t* idx,
                                                                    const float* sums, int64_t m, float world) {
    const int64_t first = (static_cast<int64_t>(blockIdx.x) * kUnionPerThread) * kUnionBlock + threadIdx.x;
    int32_t j[kUnionPerThread];
    float s[kUnionPerThread], xv[kUnionPerThread];
#pragma unroll
    for (int u = 0; u < kUnionPerThread; ++u) {
        const int64_t q = first + static_cast<int64_t>(u) * kUnionBlock;
        j[u] = q < m ? __builtin_nontemporal_load(idx + q) : -1;
        if (j[u] >= n_x) j[u] = -1;
        s[u] = q < m ? __builtin_nontemporal_load(sums + q) : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < kUnionPerThread; ++u) xv[u] = j[u] >= 0 ? x[j[u]] : 0.0f;
#pragma unroll
    for (int u = 0; u < kUnionPerThread; ++u) {
        if (j[u] >= 0) {
            const float average = s[u] / world;
            __builtin_nontemporal_store(xv[u] - average, x + j[u]);
        }
    }
}

uint32_t union_blocks(int64_t m) {
    const int64_t per_block = static_cast<int64_t>(kUnionBlock) * kUnionPerThread;
    return static_cast<uint32_t>((m + per_block - 1) / per_block);
}

}  // namespace

hipError_t launch_union_gather(float* residual, int64_t n, const int32_t* idx, int64_t m, int64_t own_first,
                               int64_t own_count, const float* own_val, float* out, hipStream_t stream) {
    if (m == 0) return hipSuccess;
    hipLaunchKernelGGL(union_gather_kernel, dim3(union_blocks(m)), dim3(kUnionBlock), 0, stream, residual, n, idx,
                       m, own_first, own_count, own_val, out);
    return hipGetLastError();
}

hipError_t launch_sparse_update(float* x, int64_t n_x, const int32_t* idx, const float* sums, int64_t m,
                                float world, hipStream_t stream) {
    if (m == 0) return hipSuccess;
    hipLaunchKernelGGL(sparse_update_kernel, dim3(union_blocks(m)), dim3(kUnionBlock), 0, stream, x, n_x, idx, sums,
                       m, world);
    return hipGetLastError();
}

}  // namespace micro
