// Internal launchers of libinferscale's kernels (host side). The C ABI in
// abi.hip validates arguments and calls these; each returns the launch
// status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "inferscale.h"

namespace is {

// Compute units of the current device (cached per device; 256 on MI355X).
int compute_units();

// retrieve.hip
hipError_t launch_scan(const void* query, const void* bank, int64_t n, int d, int nq,
                       int64_t bank_stride, int dtype, float* scores, hipStream_t st);
bool scan_mfma_applies(int64_t n, int d, int nq, int64_t bank_stride, int dtype);
// Blocks and rows per block of a matrix-core scan over `rows` rows (at most
// mfma_max_blocks() blocks; rows_per_block is a multiple of 32).
void mfma_grid(int64_t rows, int* blocks, int64_t* rows_per_block);
int mfma_max_blocks();
// Dense scores of rows [row_begin, row_end): scores[q * ld + row - row_begin].
hipError_t launch_scan_mfma(const void* query, const void* bank, int d, int nq, int64_t row_begin,
                            int64_t row_end, float* scores, int64_t ld, hipStream_t st);
// Keys above tau_keys[q * k + k - 1] of rows [row_begin, row_end), written to
// regions[q][g][rows_per_block] with counts[q][g] (g < blocks of mfma_grid).
hipError_t launch_scan_mfma_filter(const void* query, const void* bank, int d, int nq,
                                   int64_t row_begin, int64_t row_end, const uint64_t* tau_keys,
                                   int k, uint64_t* regions, uint32_t* counts, hipStream_t st);
int64_t select_chunk_len();
// The k winners of each select_chunk_len() chunk of fp32 scores [nq][n], as
// keys best first and 0-padded, to cand[q][chunk][k].
hipError_t launch_select_scores(const float* scores, int64_t n, int k, int nq, int nchunks,
                                uint64_t* cand, hipStream_t st);
// Final ranking of nlists such winner lists per query (lists[q][nlists][k]),
// for nlists * k up to the bound merge_ranked_applies checks: to out_ids /
// out_scores, or with out_keys as keys best first (0-padded) to
// out_keys[q][k].
bool merge_ranked_applies(int nlists, int k);
hipError_t launch_merge_ranked(const uint64_t* lists, int nlists, int k, int nq, int32_t* out_ids,
                               float* out_scores, uint64_t* out_keys, hipStream_t st);
// Final ranking of one chunk of fp32 scores per query (n <= select_chunk_len()).
hipError_t launch_select_small(const float* scores, int64_t n, int k, int nq, int32_t* out_ids,
                               float* out_scores, hipStream_t st);
hipError_t launch_select_keys(const uint64_t* keys, int64_t M, int k, int nq, int nchunks,
                              uint64_t* cand, int32_t* out_ids, float* out_scores, hipStream_t st);
// Final ranking from the sample winners first[q][k] and the filter survivors.
hipError_t launch_select_regions(const uint64_t* first, const uint64_t* regions,
                                 const uint32_t* counts, int G, int64_t rcap, int k, int nq,
                                 int32_t* out_ids, float* out_scores, hipStream_t st);

// place.hip
hipError_t launch_slot_map(const int32_t* ids, const int32_t* fact_lens, int32_t start_pos,
                           const int32_t* block_table, int32_t page_size, int64_t* out_slots,
                           int32_t* out_positions, int32_t* out_m, int32_t k, int32_t nq,
                           int64_t n, int64_t lens_stride, int32_t max_blocks, int32_t max_tokens,
                           int32_t reverse_rank, uint32_t* status, hipStream_t st);

// inject.hip
// Placement inputs and outputs of the fused place + inject launch.
struct PlaceArgs {
    const int32_t* block_table;  // [nq][max_blocks]
    int64_t* out_slots;          // [nq][max_tokens]
    int32_t* out_positions;      // [nq][max_tokens]
    int32_t* out_m;              // [nq]
    int32_t start_pos, page_size, max_blocks;
};
// place == nullptr: slots, positions and m are the slot map's outputs.
// Otherwise they are ignored and the launch places the facts itself.
hipError_t launch_inject(const int32_t* ids, const void* preK, const void* V, const int64_t* slots,
                         const int32_t* positions, float rope_theta, void* paged_k, void* paged_v,
                         const int64_t* fact_offsets, const int32_t* fact_lens, const int32_t* m,
                         int32_t k, int32_t nq, int64_t n, int64_t lens_stride,
                         int32_t reverse_rank, int32_t max_tokens, int32_t L, int32_t H, int32_t D,
                         int64_t T_store, int64_t num_slots, const double* inv_freq,
                         int32_t interleaved, uint32_t* status, hipStream_t st,
                         const PlaceArgs* place = nullptr);

// copy.hip: dst[i] = src[i] for i < units 16-byte units (non-temporal)
hipError_t launch_stream_copy(void* dst, const void* src, int64_t units, hipStream_t st);

// consumer.hip
int consumer_max_q_elems();
int consumer_max_group();
hipError_t launch_paged_scores(const void* q, const int32_t* qpos, const void* paged_k,
                               int32_t layer, const int32_t* block_table, int32_t page_size,
                               int32_t start_pos, const int32_t* m, float* scores, int32_t nq,
                               int32_t Hq, int32_t H, int32_t D, int64_t num_slots,
                               int32_t max_blocks, int32_t max_tokens, float rope_theta,
                               const double* inv_freq, int32_t interleaved, uint32_t* status,
                               hipStream_t st);

// ann.hip
hipError_t launch_ann_take(const int32_t* ids, int64_t row0, int nb, int R, int32_t* F,
                           hipStream_t st);
size_t ann_merge_scratch_bytes(int64_t n, int R);
hipError_t launch_ann_merge(const int32_t* F, int64_t n, int R, void* scratch, int32_t* G,
                            hipStream_t st);
hipError_t launch_ann_seeds(const void* bank, int64_t n, int d, int dtype, int n_seeds,
                            int32_t* seed_ids, void* seed_bank, hipStream_t st);
int ann_max_row_chunks();
hipError_t launch_ann_search(const void* query, int nq, const void* bank, int64_t n, int d,
                             int dtype, const int32_t* graph, int R, const int32_t* seed_ids,
                             int n_seeds, const int32_t* init_local, const float* init_score,
                             int n_init, int B, int P, int k, int max_iters, int32_t* out_ids,
                             float* out_scores, int32_t* out_iters, int32_t* out_scored,
                             uint32_t* status, hipStream_t st);

}  // namespace is
