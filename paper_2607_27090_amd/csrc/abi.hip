// C ABI of libinferscale: host-side argument validation, workspace layout and
// launch sequencing. The contract of every entry point is documented in
// include/inferscale.h.
#include <atomic>
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "launch.hpp"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

int ok() {
    g_last_error.clear();
    return IS_OK;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct RetrieveLayout {
    size_t scores_off, cand_a_off, cand_b_off, total;
    int nchunks;
};

RetrieveLayout retrieve_layout(int64_t n, int32_t k, int32_t nq) {
    RetrieveLayout lay{};
    const int64_t chunk = is::select_chunk_len();
    lay.nchunks = (int)((n + chunk - 1) / chunk);
    size_t off = 0;
    lay.scores_off = off;
    off = round_up(off + (size_t)nq * (size_t)n * sizeof(float), 256);
    lay.cand_a_off = off;
    const size_t cand = lay.nchunks > 1 ? (size_t)nq * lay.nchunks * k * sizeof(uint64_t) : 0;
    off = round_up(off + cand, 256);
    lay.cand_b_off = off;
    off = round_up(off + cand, 256);
    lay.total = off;
    return lay;
}

// Filtered matrix-core retrieval (many queries on one shared bf16 bank): the
// scores of a sample of the first S rows [nq][S], the winners of each of its
// select chunks [nq][S / chunk][k] (several chunks only), the sample's
// winners [nq][k], survivor counts [nq][G] and survivor regions [nq][G][rows
// per block], where G * rows per block <= (n - S) + 32 G (G <= the block
// bound).
struct FusedLayout {
    size_t scores_off, chunks_off, first_off, counts_off, regions_off, total;
    int64_t sample;
};

// The sample: one to four select chunks, at most a quarter of the bank. Its
// dense scan takes one row tile per block whatever its size up to a row tile
// per CU, and a larger sample leaves fewer rows to the filtered scan and a
// tighter bound (the 1M-row bank: 65,536 rows).
int64_t fused_sample(int64_t n) {
    const int64_t chunk = is::select_chunk_len();
    const int64_t c = std::min<int64_t>(4, std::max<int64_t>(1, n / (4 * chunk)));
    return c * chunk;
}

FusedLayout fused_layout(int64_t n, int32_t k, int32_t nq) {
    FusedLayout lay{};
    const int64_t S = fused_sample(n);
    const int64_t nch = S / is::select_chunk_len();
    const int64_t gmax = is::mfma_max_blocks();
    lay.sample = S;
    size_t off = 0;
    lay.scores_off = off;
    off = round_up(off + (size_t)nq * S * sizeof(float), 256);
    lay.chunks_off = off;
    if (nch > 1) off = round_up(off + (size_t)nq * nch * k * sizeof(uint64_t), 256);
    lay.first_off = off;
    off = round_up(off + (size_t)nq * k * sizeof(uint64_t), 256);
    lay.counts_off = off;
    off = round_up(off + (size_t)nq * gmax * sizeof(uint32_t), 256);
    lay.regions_off = off;
    off = round_up(off + (size_t)nq * (size_t)(n - S + 32 * gmax) * sizeof(uint64_t), 256);
    lay.total = off;
    return lay;
}

// The sample pays off once the bank is well beyond one select chunk.
bool fused_applies(int64_t n, int32_t d, int32_t nq, int64_t bank_stride, int32_t dtype) {
    return is::scan_mfma_applies(n, d, nq, bank_stride, dtype) && n > 2 * is::select_chunk_len();
}

// Enqueues the retrieval kernels (arguments already validated, workspace of
// at least retrieve_need bytes).
int enqueue_retrieve(const void* query_emb, const void* bank, int64_t n, int32_t d, int32_t k,
                     int32_t* out_ids, float* out_scores, int32_t nq, int64_t bank_stride,
                     int32_t dtype, void* workspace, hipStream_t st) {
    const RetrieveLayout lay = retrieve_layout(n, k, nq);
    const bool fused = fused_applies(n, d, nq, bank_stride, dtype);
    char* ws = (char*)workspace;
    hipError_t e;
    if (fused) {
        // 1. dense scores of the first S rows; 2. their k winners (per select
        // chunk, then merged by rank), whose k-th key bounds the answer from
        // below; 3. the rest of the bank keeps only keys above it; 4. exact
        // ranking of sample winners + survivors
        const FusedLayout fl = fused_layout(n, k, nq);
        const int64_t S = fl.sample;
        float* sc = (float*)(ws + fl.scores_off);
        uint64_t* first = (uint64_t*)(ws + fl.first_off);
        uint32_t* counts = (uint32_t*)(ws + fl.counts_off);
        uint64_t* regions = (uint64_t*)(ws + fl.regions_off);
        e = is::launch_scan_mfma(query_emb, bank, d, nq, 0, S, sc, S, st);
        if (e != hipSuccess) return fail(IS_ERR_HIP, "scan launch: %s", hipGetErrorString(e));
        const int nch = (int)(S / is::select_chunk_len());
        if (nch == 1) {
            e = is::launch_select_scores(sc, S, k, nq, 1, first, st);
        } else {
            uint64_t* chunks = (uint64_t*)(ws + fl.chunks_off);
            e = is::launch_select_scores(sc, S, k, nq, nch, chunks, st);
            if (e == hipSuccess)
                e = is::launch_merge_ranked(chunks, nch, k, nq, nullptr, nullptr, first, st);
        }
        if (e != hipSuccess) return fail(IS_ERR_HIP, "select launch: %s", hipGetErrorString(e));
        e = is::launch_scan_mfma_filter(query_emb, bank, d, nq, S, n, first, k, regions, counts,
                                        st);
        if (e != hipSuccess) return fail(IS_ERR_HIP, "scan launch: %s", hipGetErrorString(e));
        int G;
        int64_t rpb;
        is::mfma_grid(n - S, &G, &rpb);
        e = is::launch_select_regions(first, regions, counts, G, rpb, k, nq, out_ids, out_scores,
                                      st);
        if (e != hipSuccess) return fail(IS_ERR_HIP, "select launch: %s", hipGetErrorString(e));
        return ok();
    }
    float* scores = (float*)(ws + lay.scores_off);
    e = is::scan_mfma_applies(n, d, nq, bank_stride, dtype)
            ? is::launch_scan_mfma(query_emb, bank, d, nq, 0, n, scores, n, st)
            : is::launch_scan(query_emb, bank, n, d, nq, bank_stride, dtype, scores, st);
    if (e != hipSuccess) return fail(IS_ERR_HIP, "scan launch: %s", hipGetErrorString(e));
    if (lay.nchunks == 1) {
        e = is::launch_select_small(scores, n, k, nq, out_ids, out_scores, st);
        if (e != hipSuccess) return fail(IS_ERR_HIP, "select launch: %s", hipGetErrorString(e));
        return ok();
    }
    uint64_t* a = (uint64_t*)(ws + lay.cand_a_off);
    uint64_t* b = (uint64_t*)(ws + lay.cand_b_off);
    e = is::launch_select_scores(scores, n, k, nq, lay.nchunks, a, st);
    if (e != hipSuccess) return fail(IS_ERR_HIP, "select launch: %s", hipGetErrorString(e));
    if (is::merge_ranked_applies(lay.nchunks, k)) {
        e = is::launch_merge_ranked(a, lay.nchunks, k, nq, out_ids, out_scores, nullptr, st);
        if (e != hipSuccess) return fail(IS_ERR_HIP, "select launch: %s", hipGetErrorString(e));
        return ok();
    }
    int64_t M = (int64_t)lay.nchunks * k;
    const int64_t chunk = is::select_chunk_len();
    while (M > chunk) {
        const int nch = (int)((M + chunk - 1) / chunk);
        e = is::launch_select_keys(a, M, k, nq, nch, b, nullptr, nullptr, st);
        if (e != hipSuccess) return fail(IS_ERR_HIP, "select launch: %s", hipGetErrorString(e));
        uint64_t* tmp = a;
        a = b;
        b = tmp;
        M = (int64_t)nch * k;
    }
    e = is::launch_select_keys(a, M, k, nq, 1, nullptr, out_ids, out_scores, st);
    if (e != hipSuccess) return fail(IS_ERR_HIP, "select launch: %s", hipGetErrorString(e));
    return ok();
}

size_t retrieve_need(int64_t n, int32_t d, int32_t k, int32_t nq, int64_t bank_stride,
                     int32_t dtype) {
    return fused_applies(n, d, nq, bank_stride, dtype) ? fused_layout(n, k, nq).total
                                                      : retrieve_layout(n, k, nq).total;
}

// Graph build: bank rows go through exact retrieval in batches of up to
// kAnnBuildBatch queries (k = R + 1); then the forward lists, then the
// reverse-edge buckets.
constexpr int kAnnBuildBatch = 256;

struct AnnBuildLayout {
    int batch;
    size_t ids_off, fwd_off, merge_off, total;
};

AnnBuildLayout ann_build_layout(int64_t n, int32_t d, int32_t R, int32_t dtype) {
    AnnBuildLayout lay{};
    lay.batch = (int)std::min<int64_t>(kAnnBuildBatch, n);
    const int last = (int)(n - (n - 1) / lay.batch * lay.batch);
    size_t off = round_up(std::max(retrieve_need(n, d, R + 1, lay.batch, 0, dtype),
                                   retrieve_need(n, d, R + 1, last, 0, dtype)),
                          256);
    lay.ids_off = off;
    off = round_up(off + (size_t)lay.batch * (R + 1) * sizeof(int32_t), 256);
    lay.fwd_off = off;
    off = round_up(off + (size_t)n * R * sizeof(int32_t), 256);
    lay.merge_off = off;
    off = round_up(off + is::ann_merge_scratch_bytes(n, R), 256);
    lay.total = off;
    return lay;
}

// Graph search: exact retrieval of the best min(beam, n_seeds) seeds, then
// the beam search.
struct AnnSearchLayout {
    int n_init;
    size_t ids_off, scores_off, total;
};

AnnSearchLayout ann_search_layout(int32_t n_seeds, int32_t d, int32_t beam, int32_t nq,
                                  int32_t dtype) {
    AnnSearchLayout lay{};
    lay.n_init = std::min(beam, n_seeds);
    size_t off = round_up(retrieve_need(n_seeds, d, lay.n_init, nq, 0, dtype), 256);
    lay.ids_off = off;
    off = round_up(off + (size_t)nq * lay.n_init * sizeof(int32_t), 256);
    lay.scores_off = off;
    off = round_up(off + (size_t)nq * lay.n_init * sizeof(float), 256);
    lay.total = off;
    return lay;
}

int check_ann_sizes(int64_t n, int32_t d, int32_t degree, int32_t dtype) {
    if (n < 2 || n > INT32_MAX) return fail(IS_ERR_INVALID, "n=%lld must be in [2, 2^31)", (long long)n);
    if (d < 8 || d > 8192 || d % 8) return fail(IS_ERR_INVALID, "d=%d must be a multiple of 8 in [8, 8192]", d);
    if (dtype != IS_DTYPE_F32 && dtype != IS_DTYPE_BF16)
        return fail(IS_ERR_UNSUPPORTED, "dtype=%d is neither IS_DTYPE_F32 nor IS_DTYPE_BF16", dtype);
    if (degree < 1 || degree > IS_ANN_MAX_DEGREE || degree > n - 1)
        return fail(IS_ERR_INVALID, "degree=%d must be in [1, min(%d, n - 1)]", degree,
                    IS_ANN_MAX_DEGREE);
    return IS_OK;
}

// A pre-RoPE store pointer is usable by the inject kernel if it is memory of
// the current device, managed memory, or pinned host memory mapped into the
// device's address space at the same address.
int check_store_pointer(const void* p, const char* what) {
    hipPointerAttribute_t a{};
    const hipError_t e = hipPointerGetAttributes(&a, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();  // do not leave the failure for the launch check
        return fail(IS_ERR_INVALID, "%s is neither device memory nor mapped pinned host memory",
                    what);
    }
    int dev = -1;
    (void)hipGetDevice(&dev);
    switch (a.type) {
        case hipMemoryTypeDevice:
            if (a.device != dev)
                return fail(IS_ERR_INVALID, "%s is memory of device %d, not of the current device %d",
                            what, a.device, dev);
            return IS_OK;
        case hipMemoryTypeManaged:
            return IS_OK;
        case hipMemoryTypeHost:
            if (a.devicePointer != p)
                return fail(IS_ERR_INVALID,
                            "%s is pinned host memory not mapped at the same device address; pass "
                            "the address hipHostGetDevicePointer returns", what);
            return IS_OK;
        default:
            return fail(IS_ERR_INVALID, "%s is neither device memory nor mapped pinned host memory",
                        what);
    }
}

int check_retrieve_sizes(int64_t n, int32_t d, int32_t k, int32_t nq, int32_t dtype) {
    if (n < 1 || n > INT32_MAX) return fail(IS_ERR_INVALID, "n=%lld must be in [1, 2^31)", (long long)n);
    if (d < 8 || d > 8192 || d % 8) return fail(IS_ERR_INVALID, "d=%d must be a multiple of 8 in [8, 8192]", d);
    if (k < 1 || k > n || k > IS_MAX_K)
        return fail(IS_ERR_INVALID, "k=%d must be in [1, min(n, %d)]", k, IS_MAX_K);
    if (nq < 1 || nq > 65535) return fail(IS_ERR_INVALID, "nq=%d must be in [1, 65535]", nq);
    if (dtype != IS_DTYPE_F32 && dtype != IS_DTYPE_BF16)
        return fail(IS_ERR_UNSUPPORTED, "dtype=%d is neither IS_DTYPE_F32 nor IS_DTYPE_BF16", dtype);
    return IS_OK;
}

int check_retrieve_args(const void* query_emb, const void* bank, int64_t n, int32_t d, int32_t k,
                        const int32_t* out_ids, const float* out_scores, int32_t nq,
                        int64_t bank_stride, int32_t dtype) {
    if (!query_emb || !bank || !out_ids)
        return fail(IS_ERR_INVALID, "query_emb, bank and out_ids must be non-NULL");
    const int rc = check_retrieve_sizes(n, d, k, nq, dtype);
    if (rc) return rc;
    if (bank_stride < 0 || bank_stride % 8)
        return fail(IS_ERR_INVALID, "bank_stride=%lld must be >= 0 and a multiple of 8",
                    (long long)bank_stride);
    if (!aligned(query_emb, 16) || !aligned(bank, 16))
        return fail(IS_ERR_INVALID, "query_emb and bank must be 16-byte aligned");
    if (!aligned(out_ids, 4) || (out_scores && !aligned(out_scores, 4)))
        return fail(IS_ERR_INVALID, "out_ids/out_scores must be 4-byte aligned");
    return IS_OK;
}

// Scratch of is_retrieve_noalloc: one array per GPU, in the library's own
// device memory for as long as the process runs, so that the call allocates
// nothing. Host code never uses the array's name as an address (on the host
// it is only a stand-in for the symbol); it uses the device address that
// hipGetSymbolAddress returns, looked up once per device.
constexpr size_t kNoAllocScratchBytes = IS_RETRIEVE_NOALLOC_MAX_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

// Device address of `scratch` on the current device (nullptr and *err set
// on failure). Racing first calls on one device store the same address.
void* noalloc_scratch(hipError_t* err) {
    static std::atomic<void*> addr[64];
    *err = hipSuccess;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= 64) {
        *err = e != hipSuccess ? e : hipErrorInvalidDevice;
        return nullptr;
    }
    void* p = addr[dev].load(std::memory_order_acquire);
    if (p) return p;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
        *err = e != hipSuccess ? e : hipErrorInvalidSymbol;
        return nullptr;
    }
    addr[dev].store(p, std::memory_order_release);
    return p;
}

}  // namespace

namespace is {

int compute_units() {
    // cached per device; threads racing on the first call store the same value
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int cus = cached[dev].load(std::memory_order_relaxed);
    if (cus == 0) {
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
        cached[dev].store(cus, std::memory_order_relaxed);
    }
    return cus;
}

}  // namespace is

extern "C" {

const char* is_version(void) { return "inferscale-gfx950 0.1.0"; }

const char* is_last_error(void) { return g_last_error.c_str(); }

int is_retrieve_workspace_size(int64_t n, int32_t d, int32_t k, int32_t nq, int32_t dtype,
                               size_t* bytes) {
    if (!bytes) return fail(IS_ERR_INVALID, "bytes is NULL");
    *bytes = 0;
    const int rc = check_retrieve_sizes(n, d, k, nq, dtype);
    if (rc) return rc;
    size_t total = retrieve_layout(n, k, nq).total;
    // the bank layout is not known here: cover the filtered path too
    if (fused_applies(n, d, nq, 0, dtype)) total = std::max(total, fused_layout(n, k, nq).total);
    *bytes = total;
    return ok();
}

int is_retrieve(const void* query_emb, const void* bank, int64_t n, int32_t d, int32_t k,
                int32_t* out_ids, float* out_scores, int32_t nq, int64_t bank_stride,
                int32_t dtype, void* workspace, size_t workspace_bytes, void* stream) {
    const int rc = check_retrieve_args(query_emb, bank, n, d, k, out_ids, out_scores, nq,
                                       bank_stride, dtype);
    if (rc) return rc;
    const size_t need = retrieve_need(n, d, k, nq, bank_stride, dtype);
    if (!workspace || workspace_bytes < need)
        return fail(IS_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 256)) return fail(IS_ERR_INVALID, "workspace must be 256-byte aligned");

    return enqueue_retrieve(query_emb, bank, n, d, k, out_ids, out_scores, nq, bank_stride, dtype,
                            workspace, (hipStream_t)stream);
}

int is_retrieve_noalloc(const void* query_emb, const void* bank, int64_t n, int32_t d, int32_t k,
                        int32_t* out_ids, float* out_scores, int32_t nq, int64_t bank_stride,
                        int32_t dtype, void* stream) {
    const int rc = check_retrieve_args(query_emb, bank, n, d, k, out_ids, out_scores, nq,
                                       bank_stride, dtype);
    if (rc) return rc;
    const size_t need = retrieve_need(n, d, k, nq, bank_stride, dtype);
    if (need > kNoAllocScratchBytes)
        return fail(IS_ERR_WORKSPACE,
                    "these sizes need %zu bytes of scratch; is_retrieve_noalloc has %zu "
                    "(IS_RETRIEVE_NOALLOC_MAX_BYTES): call is_retrieve with a workspace",
                    need, kNoAllocScratchBytes);
    hipError_t e;
    void* ws = noalloc_scratch(&e);
    if (!ws) return fail(IS_ERR_HIP, "scratch address lookup: %s", hipGetErrorString(e));
    // every retrieval kernel writes the scratch it later reads: nothing in it
    // has to start at zero
    return enqueue_retrieve(query_emb, bank, n, d, k, out_ids, out_scores, nq, bank_stride, dtype,
                            ws, (hipStream_t)stream);
}

int is_stream_copy(void* dst, const void* src, size_t bytes, void* stream) {
    if (bytes == 0) return ok();
    if (!dst || !src) return fail(IS_ERR_INVALID, "dst and src must be non-NULL");
    if (!aligned(dst, 16) || !aligned(src, 16) || bytes % 16)
        return fail(IS_ERR_INVALID, "dst and src must be 16-byte aligned and bytes=%zu a multiple "
                    "of 16", bytes);
    const uintptr_t d0 = (uintptr_t)dst, s0 = (uintptr_t)src;
    if (d0 < s0 + bytes && s0 < d0 + bytes)
        return fail(IS_ERR_INVALID, "dst and src overlap");
    const hipError_t e = is::launch_stream_copy(dst, src, (int64_t)(bytes / 16), (hipStream_t)stream);
    if (e != hipSuccess) return fail(IS_ERR_HIP, "copy launch: %s", hipGetErrorString(e));
    return ok();
}

int is_slot_map(const int32_t* ids, const int32_t* fact_lens, int32_t start_pos,
                const int32_t* block_table, int32_t page_size, int64_t* out_slots,
                int32_t* out_positions, int32_t* out_m, int32_t k, int32_t nq, int64_t n,
                int64_t lens_stride, int32_t max_blocks, int32_t max_tokens,
                int32_t reverse_rank, uint32_t* status, void* stream) {
    if (!ids || !fact_lens || !block_table || !out_slots || !out_positions || !out_m)
        return fail(IS_ERR_INVALID, "ids, fact_lens, block_table and outputs must be non-NULL");
    if (k < 1 || k > IS_MAX_K) return fail(IS_ERR_INVALID, "k=%d must be in [1, %d]", k, IS_MAX_K);
    if (nq < 1) return fail(IS_ERR_INVALID, "nq=%d must be >= 1", nq);
    if (n < 1 || n > INT32_MAX) return fail(IS_ERR_INVALID, "n=%lld must be in [1, 2^31)", (long long)n);
    if (page_size < 1) return fail(IS_ERR_INVALID, "page_size=%d must be >= 1", page_size);
    if (start_pos < 0) return fail(IS_ERR_INVALID, "start_pos=%d must be >= 0", start_pos);
    if (max_blocks < 0 || max_tokens < 0)
        return fail(IS_ERR_INVALID, "max_blocks and max_tokens must be >= 0");
    if ((int64_t)start_pos + max_tokens > INT32_MAX)
        return fail(IS_ERR_INVALID, "start_pos + max_tokens must stay below 2^31");
    if (lens_stride < 0) return fail(IS_ERR_INVALID, "lens_stride must be >= 0");
    if (!aligned(out_slots, 8) || !aligned(ids, 4) || !aligned(fact_lens, 4) ||
        !aligned(block_table, 4) || !aligned(out_positions, 4) || !aligned(out_m, 4) ||
        (status && !aligned(status, 4)))
        return fail(IS_ERR_INVALID, "misaligned pointer argument");
    hipError_t e = is::launch_slot_map(ids, fact_lens, start_pos, block_table, page_size, out_slots,
                                       out_positions, out_m, k, nq, n, lens_stride, max_blocks,
                                       max_tokens, reverse_rank, status, (hipStream_t)stream);
    if (e != hipSuccess) return fail(IS_ERR_HIP, "slot map launch: %s", hipGetErrorString(e));
    return ok();
}

int is_inject_rotary(const int32_t* ids, const void* preK, const void* V, const int64_t* slots,
                     const int32_t* positions, float rope_theta, void* paged_k, void* paged_v,
                     const int64_t* fact_offsets, const int32_t* fact_lens, const int32_t* m,
                     int32_t k, int32_t nq, int64_t n, int64_t lens_stride, int32_t reverse_rank,
                     int32_t max_tokens, int32_t L, int32_t H, int32_t D, int64_t T_store,
                     int64_t num_slots, const double* inv_freq, int32_t pairing, uint32_t* status,
                     void* stream) {
    if (!ids || !preK || !V || !slots || !positions || !paged_k || !paged_v || !fact_offsets ||
        !fact_lens || !m)
        return fail(IS_ERR_INVALID, "every array argument except status and inv_freq must be non-NULL");
    if (k < 1 || k > IS_MAX_K) return fail(IS_ERR_INVALID, "k=%d must be in [1, %d]", k, IS_MAX_K);
    if (nq < 1 || nq > 65535) return fail(IS_ERR_INVALID, "nq=%d must be in [1, 65535]", nq);
    if (n < 1 || n > INT32_MAX) return fail(IS_ERR_INVALID, "n=%lld must be in [1, 2^31)", (long long)n);
    if (L < 1 || H < 1) return fail(IS_ERR_INVALID, "L=%d and H=%d must be >= 1", L, H);
    if (D < 16 || D % 16 || D > IS_MAX_HEAD_DIM)
        return fail(IS_ERR_UNSUPPORTED, "D=%d must be a multiple of 16 in [16, %d]", D,
                    IS_MAX_HEAD_DIM);
    if ((int64_t)H * D > (1 << 20)) return fail(IS_ERR_UNSUPPORTED, "H*D=%lld too large", (long long)H * D);
    if (T_store < 0 || num_slots < 0 || max_tokens < 0 || lens_stride < 0)
        return fail(IS_ERR_INVALID, "T_store, num_slots, max_tokens and lens_stride must be >= 0");
    if (!inv_freq && (!(rope_theta > 0.f) || !std::isfinite(rope_theta)))
        return fail(IS_ERR_INVALID, "rope_theta must be positive and finite");
    if (pairing != IS_ROPE_HALF_SPLIT && pairing != IS_ROPE_INTERLEAVED)
        return fail(IS_ERR_INVALID, "pairing=%d is neither IS_ROPE_HALF_SPLIT nor IS_ROPE_INTERLEAVED",
                    pairing);
    if (!aligned(preK, 16) || !aligned(V, 16) || !aligned(paged_k, 16) || !aligned(paged_v, 16))
        return fail(IS_ERR_INVALID, "preK, V, paged_k and paged_v must be 16-byte aligned");
    if (!aligned(slots, 8) || !aligned(fact_offsets, 8) || !aligned(ids, 4) ||
        !aligned(positions, 4) || !aligned(fact_lens, 4) || !aligned(m, 4) ||
        (status && !aligned(status, 4)) || (inv_freq && !aligned(inv_freq, 8)))
        return fail(IS_ERR_INVALID, "misaligned pointer argument");
    // the store may be device memory or device-mapped pinned host memory
    // (read over the host link); anything else would fault the kernel
    int rc = check_store_pointer(preK, "preK");
    if (rc) return rc;
    rc = check_store_pointer(V, "V");
    if (rc) return rc;
    hipError_t e = is::launch_inject(ids, preK, V, slots, positions, rope_theta, paged_k, paged_v,
                                     fact_offsets, fact_lens, m, k, nq, n, lens_stride,
                                     reverse_rank, max_tokens, L, H, D, T_store, num_slots,
                                     inv_freq, pairing, status, (hipStream_t)stream);
    if (e != hipSuccess) return fail(IS_ERR_HIP, "inject launch: %s", hipGetErrorString(e));
    return ok();
}

int is_inject(const int32_t* ids, const void* preK, const void* V, const int64_t* slots,
              const int32_t* positions, float rope_theta, void* paged_k, void* paged_v,
              const int64_t* fact_offsets, const int32_t* fact_lens, const int32_t* m,
              int32_t k, int32_t nq, int64_t n, int64_t lens_stride, int32_t reverse_rank,
              int32_t max_tokens, int32_t L, int32_t H, int32_t D, int64_t T_store,
              int64_t num_slots, uint32_t* status, void* stream) {
    return is_inject_rotary(ids, preK, V, slots, positions, rope_theta, paged_k, paged_v,
                            fact_offsets, fact_lens, m, k, nq, n, lens_stride, reverse_rank,
                            max_tokens, L, H, D, T_store, num_slots, nullptr, IS_ROPE_HALF_SPLIT,
                            status, stream);
}

int is_place_inject(const int32_t* ids, const void* preK, const void* V,
                    const int64_t* fact_offsets, const int32_t* fact_lens, int32_t start_pos,
                    const int32_t* block_table, int32_t page_size, int32_t max_blocks,
                    float rope_theta, const double* inv_freq, int32_t pairing, void* paged_k,
                    void* paged_v, int64_t* out_slots, int32_t* out_positions, int32_t* out_m,
                    int32_t k, int32_t nq, int64_t n, int64_t lens_stride, int32_t reverse_rank,
                    int32_t max_tokens, int32_t L, int32_t H, int32_t D, int64_t T_store,
                    int64_t num_slots, uint32_t* status, void* stream) {
    if (!ids || !preK || !V || !fact_offsets || !fact_lens || !block_table || !paged_k ||
        !paged_v || !out_slots || !out_positions || !out_m)
        return fail(IS_ERR_INVALID, "every array argument except status and inv_freq must be non-NULL");
    if (k < 1 || k > IS_MAX_K) return fail(IS_ERR_INVALID, "k=%d must be in [1, %d]", k, IS_MAX_K);
    if (nq < 1 || nq > 65535) return fail(IS_ERR_INVALID, "nq=%d must be in [1, 65535]", nq);
    if (n < 1 || n > INT32_MAX) return fail(IS_ERR_INVALID, "n=%lld must be in [1, 2^31)", (long long)n);
    if (page_size < 1) return fail(IS_ERR_INVALID, "page_size=%d must be >= 1", page_size);
    if (start_pos < 0) return fail(IS_ERR_INVALID, "start_pos=%d must be >= 0", start_pos);
    if (max_blocks < 0 || max_tokens < 0)
        return fail(IS_ERR_INVALID, "max_blocks and max_tokens must be >= 0");
    if ((int64_t)start_pos + max_tokens > INT32_MAX)
        return fail(IS_ERR_INVALID, "start_pos + max_tokens must stay below 2^31");
    if (L < 1 || H < 1) return fail(IS_ERR_INVALID, "L=%d and H=%d must be >= 1", L, H);
    if (D < 16 || D % 16 || D > IS_MAX_HEAD_DIM)
        return fail(IS_ERR_UNSUPPORTED, "D=%d must be a multiple of 16 in [16, %d]", D,
                    IS_MAX_HEAD_DIM);
    if ((int64_t)H * D > (1 << 20)) return fail(IS_ERR_UNSUPPORTED, "H*D=%lld too large", (long long)H * D);
    if (T_store < 0 || num_slots < 0 || lens_stride < 0)
        return fail(IS_ERR_INVALID, "T_store, num_slots and lens_stride must be >= 0");
    if (!inv_freq && (!(rope_theta > 0.f) || !std::isfinite(rope_theta)))
        return fail(IS_ERR_INVALID, "rope_theta must be positive and finite");
    if (pairing != IS_ROPE_HALF_SPLIT && pairing != IS_ROPE_INTERLEAVED)
        return fail(IS_ERR_INVALID, "pairing=%d is neither IS_ROPE_HALF_SPLIT nor IS_ROPE_INTERLEAVED",
                    pairing);
    if (!aligned(preK, 16) || !aligned(V, 16) || !aligned(paged_k, 16) || !aligned(paged_v, 16))
        return fail(IS_ERR_INVALID, "preK, V, paged_k and paged_v must be 16-byte aligned");
    if (!aligned(out_slots, 8) || !aligned(fact_offsets, 8) || !aligned(ids, 4) ||
        !aligned(out_positions, 4) || !aligned(fact_lens, 4) || !aligned(block_table, 4) ||
        !aligned(out_m, 4) || (status && !aligned(status, 4)) ||
        (inv_freq && !aligned(inv_freq, 8)))
        return fail(IS_ERR_INVALID, "misaligned pointer argument");
    int rc = check_store_pointer(preK, "preK");
    if (rc) return rc;
    rc = check_store_pointer(V, "V");
    if (rc) return rc;
    const is::PlaceArgs pl{block_table, out_slots, out_positions, out_m,
                           start_pos, page_size, max_blocks};
    hipError_t e = is::launch_inject(ids, preK, V, nullptr, nullptr, rope_theta, paged_k, paged_v,
                                     fact_offsets, fact_lens, nullptr, k, nq, n, lens_stride,
                                     reverse_rank, max_tokens, L, H, D, T_store, num_slots,
                                     inv_freq, pairing, status, (hipStream_t)stream, &pl);
    if (e != hipSuccess) return fail(IS_ERR_HIP, "place + inject launch: %s", hipGetErrorString(e));
    return ok();
}

int is_paged_scores(const void* q, const int32_t* qpos, const void* paged_k, int32_t layer,
                    const int32_t* block_table, int32_t page_size, int32_t start_pos,
                    const int32_t* m, float* scores, int32_t nq, int32_t Hq, int32_t H, int32_t D,
                    int32_t L, int64_t num_slots, int32_t max_blocks, int32_t max_tokens,
                    float rope_theta, const double* inv_freq, int32_t pairing, uint32_t* status,
                    void* stream) {
    if (!q || !qpos || !paged_k || !block_table || !m || !scores)
        return fail(IS_ERR_INVALID, "q, qpos, paged_k, block_table, m and scores must be non-NULL");
    if (nq < 1 || nq > 65535) return fail(IS_ERR_INVALID, "nq=%d must be in [1, 65535]", nq);
    if (H < 1 || Hq < H || Hq % H || Hq / H > is::consumer_max_group())
        return fail(IS_ERR_UNSUPPORTED, "Hq=%d must be a multiple of H=%d with Hq/H <= %d", Hq, H,
                    is::consumer_max_group());
    if (D < 16 || D > IS_MAX_HEAD_DIM || (D & (D - 1)))
        return fail(IS_ERR_UNSUPPORTED, "D=%d must be a power of two in [16, %d]", D,
                    IS_MAX_HEAD_DIM);
    if ((int64_t)Hq * D > is::consumer_max_q_elems())
        return fail(IS_ERR_UNSUPPORTED, "Hq*D=%lld exceeds %d", (long long)Hq * D,
                    is::consumer_max_q_elems());
    if (L < 1 || layer < 0 || layer >= L)
        return fail(IS_ERR_INVALID, "layer=%d must be in [0, L=%d)", layer, L);
    if (page_size < 1 || max_blocks < 1 || max_tokens < 0 || num_slots < 0 || start_pos < 0)
        return fail(IS_ERR_INVALID, "page_size and max_blocks must be >= 1; max_tokens, "
                                    "num_slots and start_pos >= 0");
    if (!inv_freq && (!(rope_theta > 0.f) || !std::isfinite(rope_theta)))
        return fail(IS_ERR_INVALID, "rope_theta must be positive and finite");
    if (pairing != IS_ROPE_HALF_SPLIT && pairing != IS_ROPE_INTERLEAVED)
        return fail(IS_ERR_INVALID, "pairing=%d is neither IS_ROPE_HALF_SPLIT nor IS_ROPE_INTERLEAVED",
                    pairing);
    if (!aligned(paged_k, 16) || !aligned(q, 2) || !aligned(scores, 4) || !aligned(qpos, 4) ||
        !aligned(block_table, 4) || !aligned(m, 4) || (status && !aligned(status, 4)) ||
        (inv_freq && !aligned(inv_freq, 8)))
        return fail(IS_ERR_INVALID, "misaligned pointer argument");
    hipError_t e = is::launch_paged_scores(q, qpos, paged_k, layer, block_table, page_size,
                                           start_pos, m, scores, nq, Hq, H, D, num_slots,
                                           max_blocks, max_tokens, rope_theta, inv_freq, pairing,
                                           status, (hipStream_t)stream);
    if (e != hipSuccess) return fail(IS_ERR_HIP, "paged scores launch: %s", hipGetErrorString(e));
    return ok();
}

int is_ann_build_workspace_size(int64_t n, int32_t d, int32_t degree, int32_t dtype,
                                size_t* bytes) {
    if (!bytes) return fail(IS_ERR_INVALID, "bytes is NULL");
    *bytes = 0;
    const int rc = check_ann_sizes(n, d, degree, dtype);
    if (rc) return rc;
    *bytes = ann_build_layout(n, d, degree, dtype).total;
    return ok();
}

int is_ann_build(const void* bank, int64_t n, int32_t d, int32_t degree, int32_t dtype,
                 int32_t n_seeds, int32_t* graph, int32_t* fwd, int32_t* seed_ids,
                 void* seed_bank, void* workspace, size_t workspace_bytes, void* stream) {
    if (!bank || !graph) return fail(IS_ERR_INVALID, "bank and graph must be non-NULL");
    int rc = check_ann_sizes(n, d, degree, dtype);
    if (rc) return rc;
    if (n_seeds < 0 || n_seeds > n)
        return fail(IS_ERR_INVALID, "n_seeds=%d must be in [0, n]", n_seeds);
    if (n_seeds > 0 && (!seed_ids || !seed_bank))
        return fail(IS_ERR_INVALID, "seed_ids and seed_bank must be non-NULL when n_seeds > 0");
    if (!aligned(bank, 16) || (seed_bank && !aligned(seed_bank, 16)))
        return fail(IS_ERR_INVALID, "bank and seed_bank must be 16-byte aligned");
    if (!aligned(graph, 4) || (fwd && !aligned(fwd, 4)) || (seed_ids && !aligned(seed_ids, 4)))
        return fail(IS_ERR_INVALID, "graph, fwd and seed_ids must be 4-byte aligned");
    const AnnBuildLayout lay = ann_build_layout(n, d, degree, dtype);
    if (!workspace || workspace_bytes < lay.total)
        return fail(IS_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", lay.total,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 256)) return fail(IS_ERR_INVALID, "workspace must be 256-byte aligned");

    hipStream_t st = (hipStream_t)stream;
    char* ws = (char*)workspace;
    int32_t* ids = (int32_t*)(ws + lay.ids_off);
    int32_t* F = fwd ? fwd : (int32_t*)(ws + lay.fwd_off);
    const size_t esize = dtype == IS_DTYPE_F32 ? 4 : 2;
    for (int64_t row0 = 0; row0 < n; row0 += lay.batch) {
        const int nb = (int)std::min<int64_t>(lay.batch, n - row0);
        const void* rows = (const char*)bank + (size_t)row0 * d * esize;
        rc = enqueue_retrieve(rows, bank, n, d, degree + 1, ids, nullptr, nb, 0, dtype, ws, st);
        if (rc) return rc;
        hipError_t e = is::launch_ann_take(ids, row0, nb, degree, F, st);
        if (e != hipSuccess) return fail(IS_ERR_HIP, "graph build launch: %s", hipGetErrorString(e));
    }
    hipError_t e = is::launch_ann_merge(F, n, degree, ws + lay.merge_off, graph, st);
    if (e != hipSuccess) return fail(IS_ERR_HIP, "graph merge launch: %s", hipGetErrorString(e));
    if (n_seeds > 0) {
        e = is::launch_ann_seeds(bank, n, d, dtype, n_seeds, seed_ids, seed_bank, st);
        if (e != hipSuccess) return fail(IS_ERR_HIP, "seed launch: %s", hipGetErrorString(e));
    }
    return ok();
}

static int check_ann_search_sizes(int32_t nq, int64_t n, int32_t d, int32_t dtype, int32_t degree,
                                  int32_t n_seeds, int32_t beam, int32_t width, int32_t k,
                                  int32_t max_iters) {
    int rc = check_ann_sizes(n, d, degree, dtype);
    if (rc) return rc;
    if (nq < 1 || nq > 65535) return fail(IS_ERR_INVALID, "nq=%d must be in [1, 65535]", nq);
    const int64_t row_chunks = (int64_t)d * (dtype == IS_DTYPE_F32 ? 4 : 2) / 16;
    if (row_chunks > is::ann_max_row_chunks())
        return fail(IS_ERR_UNSUPPORTED, "rows of %lld bytes exceed the search limit of %d bytes",
                    (long long)row_chunks * 16, is::ann_max_row_chunks() * 16);
    if (n_seeds < 1 || n_seeds > n)
        return fail(IS_ERR_INVALID, "n_seeds=%d must be in [1, n]", n_seeds);
    if (beam < 1 || beam > IS_ANN_MAX_BEAM)
        return fail(IS_ERR_INVALID, "beam=%d must be in [1, %d]", beam, IS_ANN_MAX_BEAM);
    if (width < 1 || width > IS_ANN_MAX_WIDTH || width * degree > IS_ANN_MAX_EXPAND)
        return fail(IS_ERR_INVALID, "width=%d must be in [1, %d] with width*degree <= %d", width,
                    IS_ANN_MAX_WIDTH, IS_ANN_MAX_EXPAND);
    if (k < 1 || k > beam) return fail(IS_ERR_INVALID, "k=%d must be in [1, beam=%d]", k, beam);
    if (max_iters < 0) return fail(IS_ERR_INVALID, "max_iters=%d must be >= 0", max_iters);
    return IS_OK;
}

int is_ann_search_workspace_size(int32_t n_seeds, int32_t d, int32_t beam, int32_t nq,
                                 int32_t dtype, size_t* bytes) {
    if (!bytes) return fail(IS_ERR_INVALID, "bytes is NULL");
    *bytes = 0;
    if (n_seeds < 1 || beam < 1 || beam > IS_ANN_MAX_BEAM || nq < 1 || nq > 65535)
        return fail(IS_ERR_INVALID, "n_seeds, beam and nq out of range");
    const int rc = check_retrieve_sizes(n_seeds, d, std::min(beam, n_seeds), nq, dtype);
    if (rc) return rc;
    *bytes = ann_search_layout(n_seeds, d, beam, nq, dtype).total;
    return ok();
}

int is_ann_search(const void* query_emb, int32_t nq, const void* bank, int64_t n, int32_t d,
                  int32_t dtype, const int32_t* graph, int32_t degree, const int32_t* seed_ids,
                  const void* seed_bank, int32_t n_seeds, int32_t beam, int32_t width, int32_t k,
                  int32_t max_iters, int32_t* out_ids, float* out_scores, int32_t* out_iters,
                  int32_t* out_scored, uint32_t* status, void* workspace, size_t workspace_bytes,
                  void* stream) {
    if (!query_emb || !bank || !graph || !seed_ids || !seed_bank || !out_ids)
        return fail(IS_ERR_INVALID,
                    "query_emb, bank, graph, seed_ids, seed_bank and out_ids must be non-NULL");
    int rc = check_ann_search_sizes(nq, n, d, dtype, degree, n_seeds, beam, width, k, max_iters);
    if (rc) return rc;
    if (!aligned(query_emb, 16) || !aligned(bank, 16) || !aligned(seed_bank, 16))
        return fail(IS_ERR_INVALID, "query_emb, bank and seed_bank must be 16-byte aligned");
    if (!aligned(graph, 4) || !aligned(seed_ids, 4) || !aligned(out_ids, 4) ||
        (out_scores && !aligned(out_scores, 4)) || (out_iters && !aligned(out_iters, 4)) ||
        (out_scored && !aligned(out_scored, 4)) || (status && !aligned(status, 4)))
        return fail(IS_ERR_INVALID, "misaligned pointer argument");
    const AnnSearchLayout lay = ann_search_layout(n_seeds, d, beam, nq, dtype);
    if (!workspace || workspace_bytes < lay.total)
        return fail(IS_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", lay.total,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 256)) return fail(IS_ERR_INVALID, "workspace must be 256-byte aligned");

    hipStream_t st = (hipStream_t)stream;
    char* ws = (char*)workspace;
    int32_t* init_ids = (int32_t*)(ws + lay.ids_off);
    float* init_scores = (float*)(ws + lay.scores_off);
    rc = enqueue_retrieve(query_emb, seed_bank, n_seeds, d, lay.n_init, init_ids, init_scores, nq,
                          0, dtype, ws, st);
    if (rc) return rc;
    hipError_t e = is::launch_ann_search(query_emb, nq, bank, n, d, dtype, graph, degree, seed_ids,
                                         n_seeds, init_ids, init_scores, lay.n_init, beam, width,
                                         k, max_iters, out_ids, out_scores, out_iters, out_scored,
                                         status, st);
    if (e != hipSuccess) return fail(IS_ERR_HIP, "graph search launch: %s", hipGetErrorString(e));
    return ok();
}

}  // extern "C"
