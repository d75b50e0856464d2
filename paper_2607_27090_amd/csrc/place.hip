// Placement and slot mapping (§5.2 Position policy: facts placed contiguously
// at cumulative offsets, the most relevant one adjacent to the query; §2.2
// paged blocks addressed through the request's block table).
//
// One 1024-thread workgroup per request: thread i loads the length of the
// fact placed i-th, a block-wide scan gives the offsets b_i and the total m,
// the request is validated as a whole, then every placed token idx gets
// position start_pos + idx and its slot from the block table. The slot of a
// token depends only on its placed index, so no per-token fact lookup is
// needed, and the block-table entries are loaded at the start, alongside the
// fact ids, instead of after the scan.
#include "common.hpp"
#include "launch.hpp"

namespace is {

constexpr int kPlaceThreads = 1024;

constexpr int kPlacePrefetch = 4;  // block-table entries each thread loads up front

__global__ __launch_bounds__(kPlaceThreads) void slot_map_kernel(
    const int32_t* __restrict__ ids, const int32_t* __restrict__ fact_lens, int32_t start_pos,
    const int32_t* __restrict__ block_table, int32_t page_size, int64_t* __restrict__ out_slots,
    int32_t* __restrict__ out_positions, int32_t* __restrict__ out_m, int32_t k, int64_t n,
    int64_t lens_stride, int32_t max_blocks, int32_t max_tokens, int32_t reverse_rank,
    uint32_t* __restrict__ status) {
    __shared__ int64_t wave_tot[kPlaceThreads / kWave];
    __shared__ uint32_t sflags;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int r = blockIdx.x;
    const int32_t* rid = ids + (int64_t)r * k;
    const int32_t* lens = fact_lens + (int64_t)r * lens_stride;
    const int32_t* bt = block_table + (int64_t)r * max_blocks;

    // independent loads first: this thread's fact id and the block-table
    // entries of the first placed tokens it will map (a token's slot depends
    // only on its placed index, never on which fact it came from)
    const int32_t c = t < k ? (reverse_rank ? rid[k - 1 - t] : rid[t]) : 0;
    int32_t pb[kPlacePrefetch];
#pragma unroll
    for (int j = 0; j < kPlacePrefetch; ++j) {
        const int64_t idx = t + (int64_t)j * kPlaceThreads;
        const int64_t blk = ((int64_t)start_pos + idx) / page_size;
        pb[j] = (idx < max_tokens && blk < max_blocks) ? bt[blk] : 0;
    }
    if (t == 0) sflags = 0;
    __syncthreads();

    uint32_t flags = 0;
    int64_t len = 0;
    if (t < k) {
        if (c < 0 || (int64_t)c >= n) {
            flags |= IS_DEV_ID_RANGE;
        } else {
            const int32_t l = lens[c];
            if (l < 0) flags |= IS_DEV_BAD_LEN;
            else len = l;
        }
    }
    if (flags) atomicOr(&sflags, flags);
    const int64_t incl = wave_incl_scan(len, lane);
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int64_t total = 0;
#pragma unroll
    for (int w = 0; w < kPlaceThreads / kWave; ++w) total += wave_tot[w];

    if (t == 0 && sflags == 0) {
        uint32_t f = 0;
        if (total > max_tokens) f |= IS_DEV_CAPACITY;
        else if (total > 0 && ((int64_t)start_pos + total - 1) / page_size >= max_blocks)
            f |= IS_DEV_BT_SHORT;
        if (f) atomicOr(&sflags, f);
    }
    __syncthreads();
    if (sflags == 0) {
        // every block the placement uses must be a real block
        bool bad = false;
#pragma unroll
        for (int j = 0; j < kPlacePrefetch; ++j)
            if (t + (int64_t)j * kPlaceThreads < total && pb[j] < 0) bad = true;
        for (int64_t idx = t + (int64_t)kPlacePrefetch * kPlaceThreads; idx < total;
             idx += kPlaceThreads)
            if (bt[((int64_t)start_pos + idx) / page_size] < 0) bad = true;
        if (bad) atomicOr(&sflags, IS_DEV_BAD_BLOCK);
    }
    __syncthreads();
    const uint32_t req_flags = sflags;
    if (req_flags) {
        if (t == 0) {
            out_m[r] = 0;
            if (status) atomicOr(status, req_flags);
        }
        return;
    }
    int64_t* slots_r = out_slots + (int64_t)r * max_tokens;
    int32_t* pos_r = out_positions + (int64_t)r * max_tokens;
#pragma unroll
    for (int j = 0; j < kPlacePrefetch; ++j) {
        const int64_t idx = t + (int64_t)j * kPlaceThreads;
        if (idx < total) {
            const int64_t p = (int64_t)start_pos + idx;
            slots_r[idx] = (int64_t)pb[j] * page_size + p % page_size;
            pos_r[idx] = (int32_t)p;
        }
    }
    for (int64_t idx = t + (int64_t)kPlacePrefetch * kPlaceThreads; idx < total;
         idx += kPlaceThreads) {
        const int64_t p = (int64_t)start_pos + idx;
        slots_r[idx] = (int64_t)bt[p / page_size] * page_size + p % page_size;
        pos_r[idx] = (int32_t)p;
    }
    if (t == 0) out_m[r] = (int32_t)total;
}

hipError_t launch_slot_map(const int32_t* ids, const int32_t* fact_lens, int32_t start_pos,
                           const int32_t* block_table, int32_t page_size, int64_t* out_slots,
                           int32_t* out_positions, int32_t* out_m, int32_t k, int32_t nq,
                           int64_t n, int64_t lens_stride, int32_t max_blocks, int32_t max_tokens,
                           int32_t reverse_rank, uint32_t* status, hipStream_t st) {
    hipLaunchKernelGGL(slot_map_kernel, dim3((unsigned)nq), dim3(kPlaceThreads), 0, st, ids,
                       fact_lens, start_pos, block_table, page_size, out_slots, out_positions,
                       out_m, k, n, lens_stride, max_blocks, max_tokens, reverse_rank, status);
    return hipGetLastError();
}

}  // namespace is
