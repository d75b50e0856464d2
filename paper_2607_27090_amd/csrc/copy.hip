// C0: a streaming device-to-device copy, the practical ceiling of HBM for a
// read-once / write-once stream. It is not a step of the method; the bench
// times it beside the inject (which moves the same kind of traffic: every
// stored byte read once, every page byte written once) to report the inject
// against what the memory system sustains, not only against the 8 TB/s spec.
//
// Grid-stride over 16-byte units with non-temporal loads and stores: at any
// moment all CUs work on neighbouring addresses (one front sweeping the
// buffers), which HBM serves better than a contiguous share per CU. Each
// thread issues kUnroll loads before its stores.
//
// Launch shape: one 256-thread workgroup per CU with 4 loads in flight per
// lane, i.e. 16 wave-wide 1 KiB loads outstanding per CU. A sweep on MI355X
// (263 MB and 1 GiB each way, caches cold) found ~16 such loads per CU best:
// 4 waves x 4 loads, 8 x 2 and 16 x 1 all reach 6.0-6.2 TB/s, while 16 waves
// x 4 loads fall to ~5.3 TB/s and 32 waves x 4 loads to ~4.5 TB/s (more
// requests in flight congest the memory system instead of filling it).
#include "common.hpp"
#include "launch.hpp"

namespace is {

constexpr int kCopyThreads = 256;
constexpr int kCopyBlocksPerCu = 1;
constexpr int kCopyUnroll = 4;

typedef uint32_t cp_u32x4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kCopyThreads) void stream_copy_kernel(
    const cp_u32x4_t* __restrict__ src, cp_u32x4_t* __restrict__ dst, int64_t units) {
    const int64_t stride = (int64_t)gridDim.x * kCopyThreads;
    int64_t i = (int64_t)blockIdx.x * kCopyThreads + threadIdx.x;
    for (; i + (kCopyUnroll - 1) * stride < units; i += kCopyUnroll * stride) {
        cp_u32x4_t v[kCopyUnroll];
#pragma unroll
        for (int u = 0; u < kCopyUnroll; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
        for (int u = 0; u < kCopyUnroll; ++u) __builtin_nontemporal_store(v[u], dst + i + u * stride);
    }
    for (; i < units; i += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

hipError_t launch_stream_copy(void* dst, const void* src, int64_t units, hipStream_t st) {
    if (units == 0) return hipSuccess;
    const int64_t per_block = (int64_t)kCopyThreads * kCopyUnroll;
    int64_t blocks = (int64_t)compute_units() * kCopyBlocksPerCu;
    const int64_t need = (units + per_block - 1) / per_block;
    if (blocks > need) blocks = need;
    hipLaunchKernelGGL(stream_copy_kernel, dim3((unsigned)blocks), dim3(kCopyThreads), 0, st,
                       (const cp_u32x4_t*)src, (cp_u32x4_t*)dst, units);
    return hipGetLastError();
}

}  // namespace is
