// Graph-ANN retrieval backend for gfx950 (§2.6: a proximity graph over the
// fact embeddings built and searched on the GPU; §6.1: inner product, 64
// neighbours per fact, beam width 64).
//
// Build. The forward list F[i] (the R best facts j != i) comes from the
// exact retrieval kernels, run with a batch of bank rows as the queries and
// k = R + 1; ann_take_kernel drops the row itself. Reverse edges: every
// (i = F[j][p], p < h = R/2) is counted per target, the counts are
// prefix-summed into bucket offsets and the (p, j) keys scattered into the
// buckets; one wave per fact then keeps its forward half, picks the R - h
// smallest (p, j) keys of its bucket whose j is not already listed (a
// running 64-wide bitonic merge held in registers, so a bucket of any size
// is ranked exactly), and fills the rest from the forward tail.
//
// Search. One 256-thread workgroup per query keeps the beam (at most 256
// 64-bit rank keys, best first, plus an expanded flag each) in LDS, with
// the query itself and an open-addressing table of the fact ids already
// scored. Each iteration takes the first `width` unexpanded beam entries,
// loads their neighbour lists (one id per thread), drops ids already in the
// table, scores the rest (16 lanes per row, every lane's 16-byte loads of
// several rows in flight at once) and merges the new keys that beat the
// beam's last entry by rank counting. Skipping a fact that was scored before
// never changes the result: a fact that is not in the beam once the beam is
// full ranks below its last entry, and that entry only moves up. The table
// is cleared and refilled with the beam whenever it would pass half full.
#include "wave.hpp"
#include "launch.hpp"

namespace is {

constexpr int kAnnMaxBeam = IS_ANN_MAX_BEAM;
constexpr int kAnnMaxWidth = IS_ANN_MAX_WIDTH;

// ---- build: forward lists --------------------------------------------------

// ids [nb][R + 1] ranked neighbours of rows row0 .. row0 + nb - 1 (each row's
// own id among them unless R + 1 rows tie above it) -> F[row][0 .. R): the
// list in order without the row itself, first R entries. One wave per row.
__global__ void ann_take_kernel(const int32_t* __restrict__ ids, int64_t row0, int nb, int R,
                                int32_t* __restrict__ F) {
    const int lane = threadIdx.x & (kWave - 1);
    const int b = blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    if (b >= nb) return;
    const int64_t self = row0 + b;
    const int32_t* src = ids + (int64_t)b * (R + 1);
    int32_t* dst = F + self * R;
    int dropped = 0;
    for (int base = 0; base <= R; base += kWave) {
        const int r = base + lane;
        const int32_t j = r <= R ? src[r] : -1;
        const bool drop = r <= R && j == self;
        const uint64_t m = __ballot(drop);
        const int pos = r - dropped - (int)lanes_below(m);
        if (r <= R && !drop && pos < R) dst[pos] = j;
        dropped += __popcll(m);
    }
}

// ---- build: reverse-edge buckets -------------------------------------------

__global__ void ann_fill_kernel(uint32_t* __restrict__ p, int64_t count, uint32_t v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < count) p[i] = v;
}

// cnt[F[j][p]] += 1 for every j and p < h.
__global__ void ann_rev_count_kernel(const int32_t* __restrict__ F, int64_t n, int R, int h,
                                     uint32_t* __restrict__ cnt) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n * h) return;
    const int64_t j = e / h;
    const int p = (int)(e - j * h);
    atomicAdd(&cnt[F[j * R + p]], 1u);
}

constexpr int kScanThreads = 1024;
constexpr int kScanItems = 4;
constexpr int kScanTile = kScanThreads * kScanItems;

// Exclusive block-wide prefix sum of one value per thread; returns the
// block total through *total.
__device__ int64_t block_excl_scan(int64_t v, int64_t* s_w, int64_t* total) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int64_t incl = wave_incl_scan(v, lane);
    if (lane == 63) s_w[w] = incl;
    __syncthreads();
    int64_t before = 0, all = 0;
    for (int i = 0; i < kScanThreads / kWave; ++i) {
        before += i < w ? s_w[i] : 0;
        all += s_w[i];
    }
    __syncthreads();
    *total = all;
    return before + incl - v;
}

__global__ __launch_bounds__(kScanThreads) void ann_scan_tiles_kernel(
    const uint32_t* __restrict__ cnt, int64_t n, int64_t* __restrict__ tile_sums) {
    __shared__ int64_t s_w[kScanThreads / kWave];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int64_t v = 0;
    for (int i = 0; i < kScanItems; ++i) v += base + i < n ? cnt[base + i] : 0;
    int64_t total;
    block_excl_scan(v, s_w, &total);
    if (threadIdx.x == 0) tile_sums[blockIdx.x] = total;
}

// In place: tile_sums becomes the exclusive prefix over tiles.
__global__ __launch_bounds__(kScanThreads) void ann_scan_sums_kernel(int64_t* __restrict__ sums,
                                                                     int64_t tiles) {
    __shared__ int64_t s_w[kScanThreads / kWave];
    int64_t carry = 0;
    for (int64_t c0 = 0; c0 < tiles; c0 += kScanThreads) {
        const int64_t i = c0 + threadIdx.x;
        const int64_t v = i < tiles ? sums[i] : 0;
        int64_t total;
        const int64_t ex = block_excl_scan(v, s_w, &total);
        if (i < tiles) sums[i] = carry + ex;
        carry += total;
    }
}

// off[i] = sum of cnt[0 .. i) for i <= n.
__global__ __launch_bounds__(kScanThreads) void ann_scan_apply_kernel(
    const uint32_t* __restrict__ cnt, int64_t n, const int64_t* __restrict__ tile_base,
    int64_t* __restrict__ off) {
    __shared__ int64_t s_w[kScanThreads / kWave];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    uint32_t c[kScanItems];
    int64_t v = 0;
    for (int i = 0; i < kScanItems; ++i) {
        c[i] = base + i < n ? cnt[base + i] : 0u;
        v += c[i];
    }
    int64_t total;
    int64_t run = tile_base[blockIdx.x] + block_excl_scan(v, s_w, &total);
    for (int i = 0; i < kScanItems; ++i) {
        if (base + i <= n) off[base + i] = run;  // off[n] = the grand total
        run += c[i];
    }
}

// entries[off[i] + slot] = (p << 32) | j for every i = F[j][p], p < h.
__global__ void ann_rev_scatter_kernel(const int32_t* __restrict__ F, int64_t n, int R, int h,
                                       const int64_t* __restrict__ off,
                                       uint32_t* __restrict__ cursor,
                                       uint64_t* __restrict__ entries) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n * h) return;
    const int64_t j = e / h;
    const int p = (int)(e - j * h);
    const int32_t i = F[j * R + p];
    const uint32_t slot = atomicAdd(&cursor[i], 1u);
    entries[off[i] + slot] = ((uint64_t)(uint32_t)p << 32) | (uint64_t)(uint32_t)j;
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
    const uint32_t lo = __shfl((uint32_t)v, src, kWave);
    const uint32_t hi = __shfl((uint32_t)(v >> 32), src, kWave);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t min64(uint64_t a, uint64_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint64_t max64(uint64_t a, uint64_t b) { return a < b ? b : a; }

// Ascending bitonic sort of one 64-bit value per lane across the wave.
__device__ __forceinline__ uint64_t wave_sort_asc(uint64_t v, int lane) {
#pragma unroll
    for (int size = 2; size <= kWave; size <<= 1) {
#pragma unroll
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            const uint64_t o = shfl_xor64(v, stride);
            const bool asc = (lane & size) == 0 || size == kWave;
            const bool lower = (lane & stride) == 0;
            v = (lower == asc) ? min64(v, o) : max64(v, o);
        }
    }
    return v;
}

// Ascending sort of a bitonic sequence held one value per lane.
__device__ __forceinline__ uint64_t wave_bitonic_merge_asc(uint64_t v, int lane) {
#pragma unroll
    for (int stride = kWave >> 1; stride > 0; stride >>= 1) {
        const uint64_t o = shfl_xor64(v, stride);
        v = (lane & stride) == 0 ? min64(v, o) : max64(v, o);
    }
    return v;
}

constexpr int kMergeWaves = 4;

// One wave per fact i: G[i] = F[i][0 .. h), then the R - h smallest bucket
// keys (p, j) whose j is not in that half, then F[i][h .. R) minus the
// reverse entries taken, until R ids are listed. R <= 128.
__global__ __launch_bounds__(kMergeWaves * kWave) void ann_merge_kernel(
    const int32_t* __restrict__ F, int64_t n, int R, const int64_t* __restrict__ off,
    const uint64_t* __restrict__ entries, int32_t* __restrict__ G) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t i = (int64_t)blockIdx.x * kMergeWaves + (threadIdx.x >> 6);
    if (i >= n) return;  // whole waves only; no block-wide barrier below
    const int h = R / 2, quota = R - h;  // h <= 64, quota <= 64
    const int32_t fwd = lane < h ? F[i * R + lane] : -1;
    const int32_t tail = lane < quota ? F[i * R + h + lane] : -1;
    const int64_t b0 = off[i], b1 = off[i + 1];
    uint64_t best = ~0ull;  // ascending across lanes: the 64 smallest so far
    for (int64_t c0 = b0; c0 < b1; c0 += kWave) {
        uint64_t v = c0 + lane < b1 ? entries[c0 + lane] : ~0ull;
        const int32_t j = (int32_t)(uint32_t)v;
        bool listed = false;
        for (int l = 0; l < h; ++l) listed |= __shfl(fwd, l, kWave) == j;
        if (listed) v = ~0ull;
        v = wave_sort_asc(v, lane);
        // the 64 smallest of two ascending runs, as a bitonic sequence
        v = min64(best, shfl64(v, kWave - 1 - lane));
        best = wave_bitonic_merge_asc(v, lane);
    }
    const bool taken = lane < quota && best != ~0ull;
    const uint64_t tmask = __ballot(taken);
    const int c = __popcll(tmask);  // taken lanes are a prefix 0 .. c-1
    const int32_t rid = (int32_t)(uint32_t)best;
    int32_t* out = G + i * R;
    if (lane < h) out[lane] = fwd;
    if (taken) out[h + lane] = rid;
    bool keep = lane < quota;
    for (int l = 0; l < c; ++l) keep &= __shfl(rid, l, kWave) != tail;
    const uint64_t kmask = __ballot(keep);
    const int pos = h + c + (int)lanes_below(kmask);
    if (keep && pos < R) out[pos] = tail;
}

// ---- seeds -----------------------------------------------------------------

// seed_ids[s] = floor(s * n / n_seeds); seed_bank[s] = bank[seed_ids[s]].
__global__ void ann_seed_kernel(const uint4* __restrict__ bank, int64_t n, int row_chunks,
                                int n_seeds, int32_t* __restrict__ seed_ids,
                                uint4* __restrict__ seed_bank) {
    const int s = blockIdx.x;
    const int64_t id = (int64_t)s * n / n_seeds;
    if (threadIdx.x == 0) seed_ids[s] = (int32_t)id;
    for (int c = threadIdx.x; c < row_chunks; c += blockDim.x)
        seed_bank[(int64_t)s * row_chunks + c] = bank[id * row_chunks + c];
}

// ---- search ----------------------------------------------------------------

constexpr int kSrchThreads = 256;
constexpr int kSrchWaves = kSrchThreads / kWave;
constexpr int kHashBits = 13;
constexpr int kHashSize = 1 << kHashBits;  // ids; cleared before passing half full
constexpr int kRowLanes = 16;              // lanes per scored row
constexpr int kRowGroups = kSrchThreads / kRowLanes;
constexpr int kQueryChunks = 512;          // 16-byte chunks of the query (8 KiB)

struct SearchShared {
    uint4 q[kQueryChunks];
    uint64_t beam[2][kAnnMaxBeam];
    uint64_t cand_key[kSrchThreads];
    uint64_t surv[kSrchThreads];
    int32_t cand_id[kSrchThreads];
    int32_t hash[kHashSize];
    int32_t exp_id[kAnnMaxWidth];
    uint32_t wcnt[kSrchWaves];
    uint8_t expanded[2][kAnnMaxBeam];
    int hcount;
    uint32_t flags;
};

__device__ __forceinline__ uint32_t hash_slot(int32_t id) {
    return ((uint32_t)id * 2654435761u) >> (32 - kHashBits);
}

// Inserts id; true if it was not in the table. The table is never more
// than half full, so the probe ends.
__device__ __forceinline__ bool hash_insert(int32_t* table, int32_t id) {
    uint32_t s = hash_slot(id);
    while (true) {
        const int32_t prev = atomicCAS(&table[s], -1, id);
        if (prev == -1) return true;
        if (prev == id) return false;
        s = (s + 1) & (kHashSize - 1);
    }
}

// Block-wide compaction: the position of this thread's item among the
// flagged items of the block, and their total. Uses sh.wcnt; ends with a
// barrier so sh.wcnt may be reused.
__device__ __forceinline__ int block_compact(bool flag, SearchShared& sh, int* total) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const uint64_t m = __ballot(flag);
    if (lane == 0) sh.wcnt[w] = (uint32_t)__popcll(m);
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < kSrchWaves; ++i) {
        before += i < w ? (int)sh.wcnt[i] : 0;
        all += (int)sh.wcnt[i];
    }
    __syncthreads();
    *total = all;
    return before + (int)lanes_below(m);
}

// Sum over the 16 lanes of a DPP row (lanes 16r .. 16r + 15); every lane of
// the row receives the same sum: pairs, quads (quad_perm), then the two
// quads of each half (row_half_mirror) and the two halves (row_mirror).
__device__ __forceinline__ float row16_sum(float v) {
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));
    return v;
}

// 16-byte dot product of a query chunk and a row chunk. bf16: four packed
// v_dot2c_f32_bf16 steps (exact products; each step adds two of them to
// the running fp32 sum, rounding to nearest even with at most about one
// ulp of error); fp32: a chain of fused multiply-adds.
__device__ __forceinline__ float dot16q(uint4 q, uint4 r, F32Tag) { return dot16(q, r, F32Tag{}); }
__device__ __forceinline__ float dot16q(uint4 q, uint4 r, BF16Tag) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    float s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, q.x),
                                              __builtin_bit_cast(bf16x2, r.x), 0.f, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, q.y),
                                        __builtin_bit_cast(bf16x2, r.y), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, q.z),
                                        __builtin_bit_cast(bf16x2, r.z), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, q.w),
                                        __builtin_bit_cast(bf16x2, r.w), s, false);
    return s;
}

template <bool QREG, int E, int N>
__device__ __forceinline__ uint4 qchunk(const SearchShared& sh, const uint4 (&qreg)[N],
                                        const int (&chunk)[E], int e) {
    if constexpr (QREG) return qreg[e];
    else return sh.q[chunk[e]];
}

// E: 16-byte chunks per lane and row (a power of two); a row has
// row_chunks <= 16 E chunks. NR rows per row group are loaded together.
// Rows of up to 2 KiB keep the lane's query chunks in registers.
template <typename Tag, int E, bool QREG = (E <= 8)>
__global__ __launch_bounds__(kSrchThreads) void ann_search_kernel(
    const uint4* __restrict__ query, const uint4* __restrict__ bank, int64_t n, int row_chunks,
    const int32_t* __restrict__ graph, int R, const int32_t* __restrict__ seed_ids,
    int n_seeds, const int32_t* __restrict__ init_local, const float* __restrict__ init_score,
    int n_init, int B, int P, int k, int max_iters, int32_t* __restrict__ out_ids,
    float* __restrict__ out_scores, int32_t* __restrict__ out_iters,
    int32_t* __restrict__ out_scored, uint32_t* __restrict__ status) {
    constexpr int NR = E >= 32 ? 1 : 32 / E;
    __shared__ SearchShared sh;
    const int t = threadIdx.x;
    const int q = blockIdx.x;
    const int g = t / kRowLanes, gl = t % kRowLanes;

    for (int c = t; c < row_chunks; c += kSrchThreads)
        sh.q[c] = query[(int64_t)q * row_chunks + c];
    for (int s = t; s < kHashSize; s += kSrchThreads) sh.hash[s] = -1;
    if (t == 0) sh.flags = 0;
    __syncthreads();
    // this lane's chunks of every row (chunks past the row's end re-read
    // chunk 0 and count for nothing) and, for short rows, its query chunks
    int chunk[E];
    bool lane_ok[E];
    uint4 qreg[QREG ? E : 1];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int ch = gl + e * kRowLanes;
        lane_ok[e] = ch < row_chunks;
        chunk[e] = lane_ok[e] ? ch : 0;
        if constexpr (QREG) qreg[e] = sh.q[chunk[e]];
    }

    // ---- the beam starts as the best seeds (re-ranked by global id) ----
    uint64_t ikey = 0;
    bool ivalid = false;
    if (t < n_init) {
        const int32_t loc = init_local[(int64_t)q * n_init + t];
        const int32_t id = loc >= 0 && loc < n_seeds ? seed_ids[loc] : -1;
        if (id >= 0 && id < n) {
            ivalid = true;
            ikey = rank_key(init_score[(int64_t)q * n_init + t], (uint32_t)id);
        } else {
            atomicOr(&sh.flags, IS_DEV_ID_RANGE);
        }
    }
    int nvalid;
    const int ipos = block_compact(ivalid, sh, &nvalid);
    if (ivalid) sh.surv[ipos] = ikey;
    __syncthreads();
    if (t < nvalid) {
        int rank = 0;
        for (int s = 0; s < nvalid; ++s) rank += sh.surv[s] > ikey;
        sh.beam[0][rank] = ikey;
        sh.expanded[0][rank] = 0;
        hash_insert(sh.hash, (int32_t)key_id(ikey));
    }
    if (t == 0) sh.hcount = nvalid;
    __syncthreads();
    int nb = nvalid, cur = 0, iters = 0, scored = 0;

    while (iters < max_iters) {
        // ---- A. the first P unexpanded entries ----
        const bool unexp = t < nb && !sh.expanded[cur][t];
        int nunexp;
        const int upos = block_compact(unexp, sh, &nunexp);
        if (nunexp == 0) break;
        const int ne = nunexp < P ? nunexp : P;
        if (unexp && upos < P) {
            sh.exp_id[upos] = (int32_t)key_id(sh.beam[cur][t]);
            sh.expanded[cur][t] = 1;
        }
        if (sh.hcount + ne * R > kHashSize / 2) {
            // the table would pass half full: keep only the beam's ids
            for (int s = t; s < kHashSize; s += kSrchThreads) sh.hash[s] = -1;
            __syncthreads();
            if (t < nb) hash_insert(sh.hash, (int32_t)key_id(sh.beam[cur][t]));
            if (t == 0) sh.hcount = nb;
        }
        __syncthreads();
        ++iters;

        // ---- B. neighbours not scored yet ----
        bool fresh = false;
        int32_t j = -1;
        if (t < ne * R) {
            const int u = t / R, r = t - u * R;
            j = graph[(int64_t)sh.exp_id[u] * R + r];
            if (j >= 0 && j < n)
                fresh = hash_insert(sh.hash, j);
            else
                atomicOr(&sh.flags, IS_DEV_ID_RANGE);
        }
        int C;
        const int cpos = block_compact(fresh, sh, &C);
        if (fresh) sh.cand_id[cpos] = j;
        if (t == 0) sh.hcount += C;
        scored += C;
        __syncthreads();

        // ---- C. scores: row group g takes rows g, g + 16, ... Every
        // load of the round is issued before the first product; slots past
        // the last candidate load nothing ----
        for (int r0 = g; r0 < C; r0 += kRowGroups * NR) {
            uint4 v[NR][E];
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                const int c = r0 + r * kRowGroups;
                if (c < C) {
                    const uint4* src = bank + (int64_t)sh.cand_id[c] * row_chunks;
#pragma unroll
                    for (int e = 0; e < E; ++e) v[r][e] = src[chunk[e]];
                }
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                const int c = r0 + r * kRowGroups;
                float s = 0.f;
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const float t_e = dot16q(qchunk<QREG>(sh, qreg, chunk, e), v[r][e], Tag{});
                    s += lane_ok[e] ? t_e : 0.f;
                }
                s = row16_sum(s);
                if (gl == 0 && c < C) sh.cand_key[c] = rank_key(s, (uint32_t)sh.cand_id[c]);
            }
        }
        __syncthreads();

        // ---- D. merge the keys that beat the beam's last entry ----
        const uint64_t floor_key = nb == B ? sh.beam[cur][B - 1] : 0ull;
        const uint64_t ck = t < C ? sh.cand_key[t] : 0ull;
        const bool enter = t < C && ck > floor_key;
        int S;
        const int spos = block_compact(enter, sh, &S);
        if (enter) sh.surv[spos] = ck;
        __syncthreads();
        const int nxt = cur ^ 1;
        if (t < S) {
            const uint64_t me = sh.surv[t];
            int rank = 0;
            for (int s = 0; s < S; ++s) rank += sh.surv[s] > me;
            int lo = 0, hi = nb;  // beam entries above me: a prefix of the beam
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (sh.beam[cur][mid] > me) lo = mid + 1; else hi = mid;
            }
            rank += lo;
            if (rank < B) {
                sh.beam[nxt][rank] = me;
                sh.expanded[nxt][rank] = 0;
            }
        }
        if (t < nb) {
            const uint64_t me = sh.beam[cur][t];
            int rank = t;
            for (int s = 0; s < S; ++s) rank += sh.surv[s] > me;
            if (rank < B) {
                sh.beam[nxt][rank] = me;
                sh.expanded[nxt][rank] = sh.expanded[cur][t];
            }
        }
        nb = nb + S < B ? nb + S : B;
        cur = nxt;
        __syncthreads();
    }

    for (int i = t; i < k; i += kSrchThreads) {
        const bool have = i < nb;
        const uint64_t key = have ? sh.beam[cur][i] : 0ull;
        out_ids[(int64_t)q * k + i] = have ? (int32_t)key_id(key) : -1;
        if (out_scores) out_scores[(int64_t)q * k + i] = have ? key_score(key) : -__builtin_inff();
    }
    if (t == 0) {
        if (out_iters) out_iters[q] = iters;
        if (out_scored) out_scored[q] = scored;
        if (status && sh.flags) atomicOr(status, sh.flags);
    }
}

// ---- launchers -------------------------------------------------------------

hipError_t launch_ann_take(const int32_t* ids, int64_t row0, int nb, int R, int32_t* F,
                           hipStream_t st) {
    hipLaunchKernelGGL(ann_take_kernel, dim3((nb + 3) / 4), dim3(4 * kWave), 0, st, ids, row0, nb,
                       R, F);
    return hipGetLastError();
}

size_t ann_merge_scratch_bytes(int64_t n, int R) {
    const int64_t tiles = (n + 1 + kScanTile - 1) / kScanTile;
    const size_t cnt = (size_t)n * sizeof(uint32_t);
    const size_t off = (size_t)(n + 1) * sizeof(int64_t);
    const size_t sums = (size_t)tiles * sizeof(int64_t);
    const size_t ent = (size_t)n * (R / 2) * sizeof(uint64_t);
    auto up = [](size_t v) { return (v + 255) / 256 * 256; };
    return up(cnt) * 2 + up(off) + up(sums) + up(ent);
}

hipError_t launch_ann_merge(const int32_t* F, int64_t n, int R, void* scratch, int32_t* G,
                            hipStream_t st) {
    const int h = R / 2;
    const int64_t tiles = (n + 1 + kScanTile - 1) / kScanTile;
    auto up = [](size_t v) { return (v + 255) / 256 * 256; };
    char* p = (char*)scratch;
    uint32_t* cnt = (uint32_t*)p;
    p += up((size_t)n * sizeof(uint32_t));
    uint32_t* cursor = (uint32_t*)p;
    p += up((size_t)n * sizeof(uint32_t));
    int64_t* off = (int64_t*)p;
    p += up((size_t)(n + 1) * sizeof(int64_t));
    int64_t* sums = (int64_t*)p;
    p += up((size_t)tiles * sizeof(int64_t));
    uint64_t* entries = (uint64_t*)p;

    const dim3 b256(256);
    const dim3 gn((unsigned)((n + 255) / 256));
    hipLaunchKernelGGL(ann_fill_kernel, gn, b256, 0, st, cnt, n, 0u);
    hipLaunchKernelGGL(ann_fill_kernel, gn, b256, 0, st, cursor, n, 0u);
    if (h > 0) {
        const dim3 ge((unsigned)((n * h + 255) / 256));
        hipLaunchKernelGGL(ann_rev_count_kernel, ge, b256, 0, st, F, n, R, h, cnt);
    }
    hipLaunchKernelGGL(ann_scan_tiles_kernel, dim3((unsigned)tiles), dim3(kScanThreads), 0, st,
                       cnt, n, sums);
    hipLaunchKernelGGL(ann_scan_sums_kernel, dim3(1), dim3(kScanThreads), 0, st, sums, tiles);
    hipLaunchKernelGGL(ann_scan_apply_kernel, dim3((unsigned)tiles), dim3(kScanThreads), 0, st,
                       cnt, n, sums, off);
    if (h > 0) {
        const dim3 ge((unsigned)((n * h + 255) / 256));
        hipLaunchKernelGGL(ann_rev_scatter_kernel, ge, b256, 0, st, F, n, R, h, off, cursor,
                           entries);
    }
    hipLaunchKernelGGL(ann_merge_kernel, dim3((unsigned)((n + kMergeWaves - 1) / kMergeWaves)),
                       dim3(kMergeWaves * kWave), 0, st, F, n, R, off, entries, G);
    return hipGetLastError();
}

hipError_t launch_ann_seeds(const void* bank, int64_t n, int d, int dtype, int n_seeds,
                            int32_t* seed_ids, void* seed_bank, hipStream_t st) {
    const int row_chunks = d * (dtype == IS_DTYPE_F32 ? 4 : 2) / 16;
    hipLaunchKernelGGL(ann_seed_kernel, dim3(n_seeds), dim3(128), 0, st, (const uint4*)bank, n,
                       row_chunks, n_seeds, seed_ids, (uint4*)seed_bank);
    return hipGetLastError();
}

int ann_max_row_chunks() { return kQueryChunks; }

template <typename Tag>
static hipError_t launch_search_tag(int E, const void* query, int nq, const void* bank, int64_t n,
                                    int row_chunks, const int32_t* graph, int R,
                                    const int32_t* seed_ids, int n_seeds,
                                    const int32_t* init_local, const float* init_score, int n_init,
                                    int B, int P, int k, int max_iters, int32_t* out_ids,
                                    float* out_scores, int32_t* out_iters, int32_t* out_scored,
                                    uint32_t* status, hipStream_t st) {
#define IS_ANN_LAUNCH(EE)                                                                         \
    hipLaunchKernelGGL((ann_search_kernel<Tag, EE>), dim3(nq), dim3(kSrchThreads), 0, st,         \
                       (const uint4*)query, (const uint4*)bank, n, row_chunks, graph, R, seed_ids, \
                       n_seeds, init_local, init_score, n_init, B, P, k, max_iters, out_ids,      \
                       out_scores, out_iters, out_scored, status)
    switch (E) {
        case 1: IS_ANN_LAUNCH(1); break;
        case 2: IS_ANN_LAUNCH(2); break;
        case 4: IS_ANN_LAUNCH(4); break;
        case 8: IS_ANN_LAUNCH(8); break;
        case 16: IS_ANN_LAUNCH(16); break;
        default: IS_ANN_LAUNCH(32); break;
    }
#undef IS_ANN_LAUNCH
    return hipGetLastError();
}

hipError_t launch_ann_search(const void* query, int nq, const void* bank, int64_t n, int d,
                             int dtype, const int32_t* graph, int R, const int32_t* seed_ids,
                             int n_seeds, const int32_t* init_local, const float* init_score,
                             int n_init, int B, int P, int k, int max_iters, int32_t* out_ids,
                             float* out_scores, int32_t* out_iters, int32_t* out_scored,
                             uint32_t* status, hipStream_t st) {
    const int row_chunks = d * (dtype == IS_DTYPE_F32 ? 4 : 2) / 16;
    int E = 1;
    while (E * kRowLanes < row_chunks) E <<= 1;
    if (dtype == IS_DTYPE_F32)
        return launch_search_tag<F32Tag>(E, query, nq, bank, n, row_chunks, graph, R, seed_ids,
                                         n_seeds, init_local, init_score, n_init, B, P, k,
                                         max_iters, out_ids, out_scores, out_iters, out_scored,
                                         status, st);
    return launch_search_tag<BF16Tag>(E, query, nq, bank, n, row_chunks, graph, R, seed_ids,
                                      n_seeds, init_local, init_score, n_init, B, P, k, max_iters,
                                      out_ids, out_scores, out_iters, out_scored, status, st);
}

}  // namespace is
