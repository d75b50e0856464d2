// Exact top-k retrieval for gfx950 (§3.2: top-k search by inner product over
// the fact embeddings; exact brute force stands in for the paper's GPU
// graph index).
//
// Two stages:
//  1. scan: s_j = <q, e_j> for every bank row, by one of
//     * scan_kernel, a bandwidth-bound GEMV: each wave streams whole rows
//       with 16-byte loads, keeps its 1-8 queries in registers and reduces
//       the per-row partial sums across the wave with a transposing
//       butterfly, so that V partial sums cost V-1 shuffles;
//     * scan_mfma_kernel (32 or more queries against one bf16 bank):
//       256-row x 256-query tiles of v_mfma_f32_32x32x16_bf16 with both
//       operands staged through LDS, writing every score or only those not
//       below a per-query threshold.
//  2. select: the k largest 64-bit rank keys (score bits, ~id) per query.
//     A 1024-thread workgroup holds up to 16384 scores in registers, bounds
//     the answer from below (a radix bracket of the thread maxima), gathers
//     the few keys above the bound and ranks them pairwise (a radix select
//     takes over when many keys tie). Larger inputs go in chunks of 16384
//     whose sorted k winners are merged by rank (each key's position in its
//     list plus binary searches in the others), or, beyond that kernel's
//     size, ranked again in chunks of keys (the smallest of k group maxima
//     bounds those); the survivors of the filtered matrix-core scan are
//     ranked by select_regions_kernel. Ties go to the lower id (score desc,
//     id asc).
#include "wave.hpp"
#include "launch.hpp"

namespace is {

// ---- scan ------------------------------------------------------------------

// Reduce V partial sums held by every lane of a wave. On return the lane
// holds the full sum of value index `*which`; lanes whose low (6 - log2 V)
// bits are zero are the unique holders.
template <int V>
__device__ __forceinline__ float wave_multi_sum(float (&a)[V], int lane, int* which) {
    int idx = 0;
#pragma unroll
    for (int half = V / 2, off = 32; half >= 1; half >>= 1, off >>= 1) {
        // the upper lane of each pair keeps the high half of the values; the
        // choice is a bit blend of two statically indexed registers (a
        // conditional pick between array elements is turned by the compiler
        // into a dynamically indexed read, i.e. a compare/select chain over
        // the whole array)
        const uint32_t m = 0u - (uint32_t)((lane & off) != 0);
#pragma unroll
        for (int i = 0; i < half; ++i) {
            const uint32_t lo = __float_as_uint(a[i]), hi = __float_as_uint(a[i + half]);
            const float keep = __uint_as_float((hi & m) | (lo & ~m));
            const float send = __uint_as_float((lo & m) | (hi & ~m));
            a[i] = keep + __shfl_xor(send, off, kWave);
        }
        idx += half & (int)m;
    }
    constexpr int kSteps = (V >= 64) ? 0 : 6 - __builtin_ctz(V);
    float v = a[0];
#pragma unroll
    for (int s = 0, off = 32 / V; s < kSteps; ++s, off >>= 1) v += __shfl_xor(v, off, kWave);
    *which = idx;
    return v;
}

// s + <a, b> over one 16-byte unit of each operand. fp32: a fused
// multiply-add chain, then added to s. bf16: v_dot2_f32_bf16 steps
// continuing the running sum (the two bf16 x bf16 products of a step are
// exact; each step adds them to the fp32 sum with one rounding), a third of
// the instructions of unpacking and multiplying element by element.
__device__ __forceinline__ float dot16_acc(uint4 a, uint4 b, float s, F32Tag) {
    return s + dot16(a, b, F32Tag{});
}
__device__ __forceinline__ float dot16_acc(uint4 a, uint4 b, float s, BF16Tag) {
    typedef __bf16 bf16x2_t2 __attribute__((ext_vector_type(2)));
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t2, a.x),
                                        __builtin_bit_cast(bf16x2_t2, b.x), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t2, a.y),
                                        __builtin_bit_cast(bf16x2_t2, b.y), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t2, a.z),
                                        __builtin_bit_cast(bf16x2_t2, b.z), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t2, a.w),
                                        __builtin_bit_cast(bf16x2_t2, b.w), s, false);
    return s;
}

// Bank rows are read once per call: non-temporal loads. From cold caches
// (the bank evicted by other work since the last request, leaving dirty lines
// in the Infinity Cache) they cut the headline retrieval from 24.3 to 18.8 us
// per request; back to back they cost nothing.
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
    typedef uint32_t u32x4_nt __attribute__((ext_vector_type(4)));
    const u32x4_nt x = __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(p));
    return make_uint4(x.x, x.y, x.z, x.w);
}

// Raw buffer descriptors: loads at byte offsets >= the descriptor's size
// read zero, which pads ragged row tiles and reduction chunks for free.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;  // gfx9-family raw buffer format word

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             kRsrcWord3);
}

__device__ __forceinline__ uint4 buffer_load16(rsrc_t r, uint32_t off) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
}
// The same with the non-temporal hint (cache-policy bit 1): bank rows are
// streamed once per call (3% less time for the 1M-row scan than ordinary
// loads); the queries, re-read for every row tile, keep ordinary loads.
__device__ __forceinline__ uint4 buffer_load16_stream(rsrc_t r, uint32_t off, uint32_t soff = 0) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, (int)soff, 2);
    return make_uint4(v[0], v[1], v[2], v[3]);
}

constexpr int kScanMaxRows = 1024;  // rows per block at most

// One block = 4 waves. blockIdx.y selects a group of NQB queries (shared
// bank) or one query and its own bank (per-query banks, NQB == 1).
template <class Tag, int CPL, int NQB, int RB>
__global__ __launch_bounds__(256) void scan_kernel(const uint4* __restrict__ query,
                                                   const uint4* __restrict__ bank, int64_t n,
                                                   int chunks, int nq, int64_t bank_stride_chunks,
                                                   int rows_per_block, float* __restrict__ scores) {
    const int lane = threadIdx.x & 63;
    // wave-uniform, so the row loops below are scalar control flow
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int q0 = blockIdx.y * NQB;
    const uint4* B = bank + (int64_t)blockIdx.y * bank_stride_chunks;

    uint4 qr[NQB][CPL];
#pragma unroll
    for (int qq = 0; qq < NQB; ++qq)
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const int ci = lane + c * kWave;
            qr[qq][c] = (q0 + qq < nq && ci < chunks) ? query[(int64_t)(q0 + qq) * chunks + ci]
                                                     : make_uint4(0, 0, 0, 0);
        }

    const int64_t tile0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t tile1 = min(n, tile0 + rows_per_block);
    int64_t base = tile0 + (int64_t)wave * RB;
    constexpr int64_t kStep = 4 * RB;  // rows between a wave's batches

    // sum of RB rows x NQB queries, reduced across the wave; the lanes whose
    // low bits are zero hand (query, row offset, score) to put()
    auto reduce_rows = [&](uint4 (&v)[RB][CPL], auto&& put) {
        float part[NQB * RB];
#pragma unroll
        for (int qq = 0; qq < NQB; ++qq)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                float s = 0.f;
#pragma unroll
                for (int c = 0; c < CPL; ++c) s = dot16_acc(v[rb][c], qr[qq][c], s, Tag{});
                part[qq * RB + rb] = s;
            }
        int which;
        const float tot = wave_multi_sum<NQB * RB>(part, lane, &which);
        constexpr int kLowBits = (NQB * RB >= 64) ? 0 : 6 - __builtin_ctz(NQB * RB);
        if ((lane & ((1 << kLowBits) - 1)) == 0) put(which / RB, which % RB, tot);
    };

    if constexpr (NQB == 1) {
        // One query per block (the single-query bank, per-user banks): the
        // grid is fine-grained (a few batches per wave, many waves per CU),
        // so each batch is loaded, reduced and stored in turn.
        for (; base < tile1; base += kStep) {
            uint4 v[RB][CPL];
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int c = 0; c < CPL; ++c) {
                    const int ci = lane + c * kWave;
                    const int64_t row = base + rb;
                    v[rb][c] = (row < tile1 && ci < chunks) ? load_stream(B + row * chunks + ci)
                                                            : make_uint4(0, 0, 0, 0);
                }
            reduce_rows(v, [&](int qq, int rb, float tot) {
                const int64_t row = base + rb;
                if (row < tile1 && q0 + qq < nq) scores[(int64_t)(q0 + qq) * n + row] = tot;
            });
        }
    } else {
        // Several queries per block: a coarse grid whose waves stream many
        // batches each. The wave's next batch is loaded before the current
        // one is reduced, so its loads stay in flight through the arithmetic.
        //
        // Loads go through one buffer descriptor for the block's rows (at
        // most kScanMaxRows rows of at most 16 KiB): a row's byte offset is a
        // wave-uniform scalar and each lane adds a fixed unit offset, so a
        // load needs no address registers of its own. Every load is issued
        // unconditionally, so the loads of a batch go out together: a row
        // past the share re-reads the share's last row and a unit past the
        // row re-reads the row's last unit (zeroed before use: its query
        // unit is zero, and the bank unit need not be finite).
        //
        // The scores are collected in shared memory and written out at the
        // end, row-contiguous per query: a global store inside the loop
        // would make it wait for the prefetched loads each time (a store's
        // registers are reused only after it completes, and loads and stores
        // complete in one counter).
        __shared__ float s_out[NQB][kScanMaxRows];
        const rsrc_t brs = make_rsrc(B + tile0 * chunks, (uint32_t)((tile1 - tile0) * chunks * 16));
        uint32_t col_off[CPL], col_mask[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            col_off[c] = (uint32_t)min(lane + c * kWave, chunks - 1) * 16u;
            col_mask[c] = lane + c * kWave < chunks ? ~0u : 0u;
        }
        auto load_rows = [&](int64_t b, uint4 (&v)[RB][CPL]) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                const uint32_t roff =
                    (uint32_t)(min(b + rb, tile1 - 1) - tile0) * (uint32_t)chunks * 16u;
#pragma unroll
                for (int c = 0; c < CPL; ++c) v[rb][c] = buffer_load16_stream(brs, col_off[c], roff);
            }
        };
        auto reduce_batch = [&](int64_t b, uint4 (&v)[RB][CPL]) {
#pragma unroll
            for (int c = 0; c < CPL; ++c)
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) {
                    v[rb][c].x &= col_mask[c];
                    v[rb][c].y &= col_mask[c];
                    v[rb][c].z &= col_mask[c];
                    v[rb][c].w &= col_mask[c];
                }
            reduce_rows(v, [&](int qq, int rb, float tot) {
                if (b + rb < tile1) s_out[qq][b + rb - tile0] = tot;
            });
        };
        // The last batch is reduced on a path of its own, so that on every
        // path the number of loads in flight is fixed and the wait before
        // each reduction covers exactly its own batch.
        if (base < tile1) {
            uint4 v0[RB][CPL], v1[RB][CPL];
            load_rows(base, v0);
            for (;;) {
                if (base + kStep >= tile1) {
                    reduce_batch(base, v0);
                    break;
                }
                load_rows(base + kStep, v1);
                // keep the scheduler from sinking the loads below the arithmetic
                __builtin_amdgcn_sched_barrier(0);
                reduce_batch(base, v0);
                base += kStep;
                if (base + kStep >= tile1) {
                    reduce_batch(base, v1);
                    break;
                }
                load_rows(base + kStep, v0);
                __builtin_amdgcn_sched_barrier(0);
                reduce_batch(base, v1);
                base += kStep;
            }
        }
        __syncthreads();
        const int rows = (int)(tile1 - tile0);
#pragma unroll
        for (int qq = 0; qq < NQB; ++qq) {
            if (q0 + qq >= nq) break;
            float* out = scores + (int64_t)(q0 + qq) * n + tile0;
            for (int r = threadIdx.x; r < rows; r += 256) out[r] = s_out[qq][r];
        }
    }
}

template <class Tag, int CPL, int NQB>
static hipError_t launch_scan_t(const void* query, const void* bank, int64_t n, int chunks, int nq,
                                int64_t bank_stride_chunks, float* scores, hipStream_t st) {
    constexpr int RB = (CPL <= 2) ? 4 : (CPL <= 4 ? 2 : 1);
    const int groups = bank_stride_chunks ? nq : (nq + NQB - 1) / NQB;
    // aim for ~4096 blocks over the whole grid (at least 4 RB rows each: the
    // 10,000-row bank of one query gets 1,250); ~512 when a row load serves
    // 4 or 8 queries (fewer, longer-running waves keep fewer rows in flight
    // per CU, which streams faster: 70B shape, 8 queries, 23% less time).
    // 64 per-user banks of 2,000 rows: 4,032 blocks, 3% less time than 2,048
    const int64_t target = NQB >= 4 ? 512 : 4096;
    int64_t rpb = (n * groups + target - 1) / target;
    rpb = ((rpb + 4 * RB - 1) / (4 * RB)) * (4 * RB);
    if (rpb < 4 * RB) rpb = 4 * RB;
    if (rpb > 1024) rpb = 1024;
    const int64_t gx = (n + rpb - 1) / rpb;
    dim3 grid((unsigned)gx, (unsigned)groups);
    hipLaunchKernelGGL((scan_kernel<Tag, CPL, NQB, RB>), grid, dim3(256), 0, st,
                       (const uint4*)query, (const uint4*)bank, n, chunks, nq, bank_stride_chunks,
                       (int)rpb, scores);
    return hipGetLastError();
}

hipError_t launch_scan(const void* query, const void* bank, int64_t n, int d, int nq,
                       int64_t bank_stride, int dtype, float* scores, hipStream_t st) {
    const int esz = dtype == 0 ? 4 : 2;
    const int chunks = d * esz / 16;
    const int64_t bsc = bank_stride * esz / 16;
    const int cpl = (chunks + kWave - 1) / kWave;
    // A shared bank serves several queries per block so each loaded row is
    // reused from registers: 8 queries while a row takes <= 2 loads per lane,
    // 4 while it takes <= 4; beyond that one query per block.
    const bool multi = bsc == 0 && nq > 1;
#define IS_SCAN(TAG)                                                                          \
    do {                                                                                      \
        if (multi && cpl <= 1) return launch_scan_t<TAG, 1, 8>(query, bank, n, chunks, nq, bsc, scores, st); \
        if (multi && cpl <= 2) return launch_scan_t<TAG, 2, 8>(query, bank, n, chunks, nq, bsc, scores, st); \
        if (multi && cpl <= 3) return launch_scan_t<TAG, 3, 4>(query, bank, n, chunks, nq, bsc, scores, st); \
        if (multi && cpl <= 4) return launch_scan_t<TAG, 4, 4>(query, bank, n, chunks, nq, bsc, scores, st); \
        if (cpl <= 1) return launch_scan_t<TAG, 1, 1>(query, bank, n, chunks, nq, bsc, scores, st);          \
        if (cpl <= 2) return launch_scan_t<TAG, 2, 1>(query, bank, n, chunks, nq, bsc, scores, st);          \
        if (cpl <= 3) return launch_scan_t<TAG, 3, 1>(query, bank, n, chunks, nq, bsc, scores, st);          \
        if (cpl <= 4) return launch_scan_t<TAG, 4, 1>(query, bank, n, chunks, nq, bsc, scores, st);          \
        if (cpl <= 8) return launch_scan_t<TAG, 8, 1>(query, bank, n, chunks, nq, bsc, scores, st);          \
        return launch_scan_t<TAG, 16, 1>(query, bank, n, chunks, nq, bsc, scores, st);                       \
    } while (0)
    if (dtype == 0) IS_SCAN(F32Tag);
    IS_SCAN(BF16Tag);
#undef IS_SCAN
}

// ---- batched scan on the matrix cores (many queries, one shared bf16 bank) ----
//
// Scores for nq queries against one bank form the product bank (n x d) times
// queries^T (d x nq). A persistent 512-thread block owns one contiguous,
// equal share of the bank rows and walks it in tiles of 256 rows x 256
// queries; each wave accumulates kMmWaveRows rows x 128 queries with
// v_mfma_f32_32x32x16_bf16 (exact bf16 products, fp32 sums). The reduction
// dimension advances in chunks of 64: each chunk of the bank tile (32 KiB)
// and of the query tile (32 KiB) is staged in shared memory, double
// buffered. The bank is the only operand that comes from HBM (the query
// tile stays in L2), so every thread keeps kMmDepth bank chunks in flight
// in registers, and the pipeline runs on across tile boundaries. Rows are
// 128 bytes in shared memory and the eight 16-byte units of a row are
// XOR-swizzled (swz below), so the rows a fragment read touches fall in
// distinct banks.
//
// Two epilogues per finished tile:
//  * dense: every score is stored, scores[q * ld + (row - row_begin)];
//  * filter: only keys whose score is not below the score of a per-query
//    threshold key tau_q are kept. tau_q is the k-th best key of a row sample,
//    so every key of the exact top-k outside the sample is above it: the
//    top-k of the sample's top-k plus these survivors is the exact top-k.
//    Survivors of block g and query q go to their own region [q][g] of
//    capacity rows_per_block, which cannot overflow.

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kMmRows = 256;     // bank rows per tile
constexpr int kMmQ = 256;        // queries per tile
constexpr int kMmK = 64;         // reduction chunk
constexpr int kMmWaveRows = 64;                  // bank rows per wave (x 128 queries)
constexpr int kMmFragA = kMmWaveRows / 32;        // 32-row fragments per wave
constexpr int kMmRowGroups = kMmRows / kMmWaveRows;
constexpr int kMmThreads = kMmRowGroups * 2 * 64;  // row groups x 2 query groups
constexpr int kMmDepth = 2;      // chunks in flight per thread
constexpr int kMmSlots = kMmRows * 8 / kMmThreads;  // 16-byte staging slots per thread
constexpr int kMmMaxBlocks = 1024;

constexpr uint32_t kOutOfRange = 0x80000000u;  // beyond any descriptor here (<= 4 MiB)

// Shared-memory swizzle of the eight 16-byte units of a 128-byte row: any 8
// consecutive rows, and the 8 even or 8 odd rows of any 16 consecutive rows,
// put a given unit in distinct 16-byte bank groups, so fragment reads of 32
// consecutive rows are conflict-free with 128- and 256-byte bank cycles.
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

template <bool FILTER>
__global__ __launch_bounds__(kMmThreads) void scan_mfma_kernel(
    const uint4* __restrict__ bank, const uint4* __restrict__ query, int d, int nq,
    int64_t row_begin, int64_t row_end, int64_t rows_per_block, float* __restrict__ scores,
    int64_t ld, const uint64_t* __restrict__ tau_keys, int k, uint64_t* __restrict__ regions,
    uint32_t* __restrict__ counts) {
    __shared__ uint4 sA[2][kMmRows * 8];
    __shared__ uint4 sB[2][kMmQ * 8];
    __shared__ uint32_t s_cnt[FILTER ? kMmQ : 1];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int wr = wave % kMmRowGroups, wq = wave / kMmRowGroups;
    const int q0 = blockIdx.y * kMmQ;
    const int G = gridDim.x;
    const int units = d >> 3;                 // 16-byte units per row
    // reduction chunks per tile, padded to a multiple of the prefetch depth
    // (padding chunks read as zero)
    const int nk = ((d + kMmK - 1) / kMmK + kMmDepth - 1) / kMmDepth * kMmDepth;
    const int64_t blk0 = row_begin + (int64_t)blockIdx.x * rows_per_block;
    const int64_t blk1 = min(row_end, blk0 + rows_per_block);

    if (FILTER && t < kMmQ) s_cnt[t] = 0;
    if (blk0 >= blk1) {
        // an empty share still reports its (zero) survivor counts
        if (FILTER && t < kMmQ && q0 + t < nq) counts[(int64_t)(q0 + t) * G + blockIdx.x] = 0;
        return;
    }
    const int nrows = (int)(blk1 - blk0);  // rows of this block's share
    const int ntiles = (nrows + kMmRows - 1) / kMmRows;
    const int steps = ntiles * nk;  // (tile, chunk) pairs of this block, tile major

    // staging slot i = t + kMmThreads j (j < kMmSlots) holds row i / 8 =
    // t / 8 + 32 j, unit i % 8 = t % 8 of a chunk; bank and query tiles use
    // the same offsets
    constexpr int kRowStep = kMmThreads / 8;
    const int r_t = t >> 3, u_t = t & 7;
    auto chunk_off = [&](int kc, int j) -> uint32_t {
        const int gu = kc * 8 + u_t;
        return gu < units ? (uint32_t)(((r_t + kRowStep * j) * units + gu) * 16) : kOutOfRange;
    };
    const rsrc_t qsrc = make_rsrc(query + (int64_t)q0 * units,
                                  (uint32_t)(min(nq - q0, kMmQ) * units * 16));
    auto load_a = [&](int s, uint4 (&dst)[kMmSlots]) {
        const int sc = min(s, steps - 1);
        const int tile = sc / nk, kc = sc - tile * nk;
        const int64_t r0 = blk0 + (int64_t)tile * kMmRows;
        const int64_t rows = min_i64(blk1 - r0, kMmRows);
        const rsrc_t asrc = make_rsrc(bank + r0 * units, (uint32_t)(rows * units * 16));
#pragma unroll
        for (int j = 0; j < kMmSlots; ++j) dst[j] = buffer_load16_stream(asrc, chunk_off(kc, j));
    };
    auto load_b = [&](int s, uint4 (&dst)[kMmSlots]) {
        const int kc = min(s, steps - 1) % nk;
#pragma unroll
        for (int j = 0; j < kMmSlots; ++j) dst[j] = buffer_load16(qsrc, chunk_off(kc, j));
    };
    auto store_chunk = [&](int buf, const uint4 (&a)[kMmSlots], const uint4 (&b)[kMmSlots]) {
#pragma unroll
        for (int j = 0; j < kMmSlots; ++j) {
            const int r = r_t + kRowStep * j;
            sA[buf][r * 8 + (u_t ^ swz(r))] = a[j];
            sB[buf][r * 8 + (u_t ^ swz(r))] = b[j];
        }
    };

    f32x16_t acc[kMmFragA][4];

    // every fragment row / column this lane reads is = lane (mod 32), so one
    // swizzled unit offset per reduction step serves all of them
    const uint4* pa = &sA[0][(wr * kMmWaveRows + (lane & 31)) * 8];
    const uint4* pb = &sB[0][(wq * 128 + (lane & 31)) * 8];
    auto compute = [&](int buf, auto&& after_ks) {
#pragma unroll
        for (int ks = 0; ks < kMmK / 16; ++ks) {
            const int off = buf * (kMmRows * 8) + ((ks * 2 + (lane >> 5)) ^ swz(lane & 31));
            bf16x8_t fa[kMmFragA], fb[4];
#pragma unroll
            for (int a = 0; a < kMmFragA; ++a)
                fa[a] = __builtin_bit_cast(bf16x8_t, pa[a * 32 * 8 + off]);
#pragma unroll
            for (int b = 0; b < 4; ++b) fb[b] = __builtin_bit_cast(bf16x8_t, pb[b * 32 * 8 + off]);
#pragma unroll
            for (int a = 0; a < kMmFragA; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[a], fb[b], acc[a][b], 0, 0, 0);
            after_ks(ks);
        }
        // instruction order per reduction step: its fragment reads, then the
        // two staging writes of after_ks spread among its matrix ops (left to
        // itself the scheduler gathers all writes after the last matrix op,
        // where nothing overlaps them)
#pragma unroll
        for (int ks = 0; ks < kMmK / 16; ++ks) {
            __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);  // fragment reads
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // matrix ops
            __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // staging writes
            __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);  // matrix ops
            __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // staging writes
            __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);  // matrix ops
        }
    };

    // filter: the threshold scores of the lane's 4 query columns
    float tau_s[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        const int q = q0 + wq * 128 + b * 32 + (lane & 31);
        tau_s[b] = (FILTER && q < nq) ? key_score(tau_keys[(int64_t)q * k + (k - 1)]) : 0.f;
    }

    // epilogue of a finished tile: lane holds query column (lane & 31) of each
    // 32x32 tile and, for element e, row 8 (e / 4) + 4 (lane / 32) + e % 4
    auto epilogue = [&](int tile) {
        const int64_t r0 = blk0 + (int64_t)tile * kMmRows;
#pragma unroll
        for (int a = 0; a < kMmFragA; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int qq = wq * 128 + b * 32 + (lane & 31);
                const int q = q0 + qq;
                const f32x16_t& v = acc[a][b];
                if (FILTER) {
                    // keep every key whose score is not below tau's: a superset
                    // of the keys above tau (also when a score or tau is NaN),
                    // and any superset of the top-k ranks to the same top-k.
                    // The block maximum (NaN-ignoring) rules out a whole 32x32
                    // block at once; a NaN score is only needed when tau is NaN.
                    float mx = v[0];
#pragma unroll
                    for (int e = 1; e < 16; ++e) mx = fmaxf(mx, v[e]);
                    if (!(mx < tau_s[b]) && q < nq) {
#pragma unroll
                        for (int e = 0; e < 16; ++e) {
                            const int rr = tile * kMmRows + wr * kMmWaveRows + a * 32 + 8 * (e >> 2) +
                                           4 * (lane >> 5) + (e & 3);  // row within the share
                            if (!(v[e] < tau_s[b]) && rr < nrows) {
                                // the region address is formed here only (the
                                // empty asm keeps it from being hoisted into
                                // registers live across the whole scan)
                                int ql = q;
                                asm volatile("" : "+v"(ql));
                                uint64_t* reg =
                                    regions + ((int64_t)ql * G + blockIdx.x) * rows_per_block;
                                const uint32_t pos = atomicAdd(&s_cnt[qq], 1u);
                                reg[pos] = rank_key(v[e], (uint32_t)(blk0 + rr));
                            }
                        }
                    }
                    // one 32x32 block at a time: keeps the accumulators from
                    // being read out (and spilled) all at once
                    __builtin_amdgcn_sched_barrier(0);
                } else {
                    if (q >= nq) continue;
                    float* out = scores + (int64_t)q * ld - row_begin;
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int64_t row = r0 + wr * kMmWaveRows + a * 32 + 8 * g + 4 * (lane >> 5);
                        if (row + 3 < blk1 && ((ld | (row - row_begin)) & 3) == 0) {
                            *(float4*)(out + row) =
                                make_float4(v[4 * g], v[4 * g + 1], v[4 * g + 2], v[4 * g + 3]);
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                if (row + e < blk1) out[row + e] = v[4 * g + e];
                        }
                    }
                }
            }
    };

    // pipeline over the block's (tile, chunk) steps s = tile * nk + chunk:
    // chunk s is in shared memory while the bank and query parts of chunks
    // s+1 .. s+kMmDepth are in flight in ra[] / rb[]. Loads complete in issue
    // order, so both parts of a chunk are issued together, kMmDepth steps
    // before they are staged. Chunk s lives in slot s % kMmDepth, and nk is a
    // multiple of kMmDepth, so every register index is static.
    uint4 ra[kMmDepth][kMmSlots], rb[kMmDepth][kMmSlots];
#pragma unroll
    for (int j = 0; j < kMmDepth; ++j) {
        load_b(j, rb[j]);
        load_a(j, ra[j]);
    }
    store_chunk(0, ra[0], rb[0]);
    __syncthreads();
    for (int tile = 0; tile < ntiles; ++tile) {
#pragma unroll
        for (int a = 0; a < kMmFragA; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b) acc[a][b] = f32x16_t{};
        for (int kc0 = 0; kc0 < nk; kc0 += kMmDepth) {
#pragma unroll
            for (int p = 0; p < kMmDepth; ++p) {
                const int s = tile * nk + kc0 + p;
                const int buf = s & 1;
                load_b(s + kMmDepth, rb[p]);
                load_a(s + kMmDepth, ra[p]);
                // issue the loads before this step's matrix work (the
                // scheduler would otherwise sink them below it)
                __builtin_amdgcn_sched_barrier(0);
                // the next chunk is staged slot by slot between this chunk's
                // reduction steps, so its shared-memory writes overlap the
                // matrix work (the buffer written was last read before the
                // previous barrier)
                compute(buf, [&](int ks) {
                    static_assert(kMmSlots == kMmK / 16, "one staging slot per reduction step");
                    const int r = r_t + kRowStep * ks;
                    sA[buf ^ 1][r * 8 + (u_t ^ swz(r))] = ra[(p + 1) % kMmDepth][ks];
                    sB[buf ^ 1][r * 8 + (u_t ^ swz(r))] = rb[(p + 1) % kMmDepth][ks];
                });
                __syncthreads();
            }
        }
        epilogue(tile);
    }
    if (FILTER) {
        __syncthreads();  // every wave's survivors are counted
        if (t < kMmQ && q0 + t < nq) counts[(int64_t)(q0 + t) * G + blockIdx.x] = s_cnt[t];
    }
}

bool scan_mfma_applies(int64_t n, int d, int nq, int64_t bank_stride, int dtype) {
    return dtype == IS_DTYPE_BF16 && bank_stride == 0 && nq >= 32 && d >= 64;
}

void mfma_grid(int64_t rows, int* blocks, int64_t* rows_per_block) {
    int64_t g = (rows + kMmRows - 1) / kMmRows;
    const int64_t cap = compute_units() < kMmMaxBlocks ? compute_units() : kMmMaxBlocks;
    if (g > cap) g = cap;
    if (g < 1) g = 1;
    int64_t rpb = (rows + g - 1) / g;
    rpb = (rpb + 31) / 32 * 32;
    *blocks = (int)g;
    *rows_per_block = rpb;
}

int mfma_max_blocks() { return kMmMaxBlocks; }

hipError_t launch_scan_mfma(const void* query, const void* bank, int d, int nq, int64_t row_begin,
                            int64_t row_end, float* scores, int64_t ld, hipStream_t st) {
    int G;
    int64_t rpb;
    mfma_grid(row_end - row_begin, &G, &rpb);
    dim3 grid((unsigned)G, (unsigned)((nq + kMmQ - 1) / kMmQ));
    hipLaunchKernelGGL(scan_mfma_kernel<false>, grid, dim3(kMmThreads), 0, st, (const uint4*)bank,
                       (const uint4*)query, d, nq, row_begin, row_end, rpb, scores, ld,
                       (const uint64_t*)nullptr, 1, (uint64_t*)nullptr, (uint32_t*)nullptr);
    return hipGetLastError();
}

hipError_t launch_scan_mfma_filter(const void* query, const void* bank, int d, int nq,
                                   int64_t row_begin, int64_t row_end, const uint64_t* tau_keys,
                                   int k, uint64_t* regions, uint32_t* counts, hipStream_t st) {
    int G;
    int64_t rpb;
    mfma_grid(row_end - row_begin, &G, &rpb);
    dim3 grid((unsigned)G, (unsigned)((nq + kMmQ - 1) / kMmQ));
    hipLaunchKernelGGL(scan_mfma_kernel<true>, grid, dim3(kMmThreads), 0, st, (const uint4*)bank,
                       (const uint4*)query, d, nq, row_begin, row_end, rpb, (float*)nullptr,
                       (int64_t)0, tau_keys, k, regions, counts);
    return hipGetLastError();
}

// ---- select ------------------------------------------------------------------

constexpr int kSelThreads = 1024;
constexpr int kSelKpt = 16;

constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kSelCap = 2048;      // candidates kept in shared memory
constexpr int kSelRankMax = 512;   // largest candidate set ranked pairwise

struct SelShared {
    uint64_t cand[kSelCap];
    uint64_t group[IS_MAX_K];
    uint64_t sel[IS_MAX_K];
    uint32_t hist[256];
    uint32_t wcnt[kSelWaves];
    uint64_t tau;
    uint32_t count;
    uint32_t digit;
    uint32_t above;
};

__device__ __forceinline__ uint64_t wave_min64(uint64_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint64_t o = shfl_xor64(v, off);
        v = o < v ? o : v;
    }
    return v;
}

__device__ __forceinline__ uint64_t wave_or64(uint64_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v |= shfl_xor64(v, off);
    return v;
}

// Exact rank of each of sh.cand[0 .. cand_total) (the number of larger
// candidates; keys are distinct), writing the `want` best to sh.sel in rank
// order: S consecutive lanes share a candidate and split its comparisons.
// Ends with a barrier.
__device__ __forceinline__ void rank_candidates(uint32_t cand_total, int want, SelShared& sh) {
    const int t = threadIdx.x;
    uint32_t S = 1;
    while (S < 16 && 2 * S * cand_total <= (uint32_t)kSelThreads) S <<= 1;
    const uint32_t part = (uint32_t)t & (S - 1);
    for (uint32_t c = (uint32_t)t / S; c < cand_total; c += kSelThreads / S) {
        const uint64_t me = sh.cand[c];
        uint32_t rank = 0;
        uint32_t j = part;
        for (; j + 3 * S < cand_total; j += 4 * S)
            rank += (sh.cand[j] > me) + (sh.cand[j + S] > me) + (sh.cand[j + 2 * S] > me) +
                    (sh.cand[j + 3 * S] > me);
        for (; j < cand_total; j += S) rank += sh.cand[j] > me;
        for (uint32_t off = 1; off < S; off <<= 1) rank += __shfl_xor(rank, (int)off, kWave);
        if (part == 0 && rank < (uint32_t)want) sh.sel[rank] = me;
    }
    __syncthreads();
}

// One block selects the `want` = min(k, valid keys) largest keys held in its
// registers (kSelKpt per thread; keys are distinct: the low word is ~id, and
// 0 marks an empty entry). On return sh.sel[0 .. want) holds them, best
// first, and every thread has passed a barrier after they were written.
//  1. Lower bound: thread t folds its keys' maximum into group t mod want;
//     the smallest group maximum tau has at least `want` keys >= it (one per
//     group), so the answer lies among the keys >= tau, typically a few
//     times `want` of them.
//  2. The candidates are compacted with wave ballots (no atomics) and, when
//     few, ranked exactly by pairwise comparison, which also orders them;
//     otherwise a radix select over the candidates picks the `want` largest
//     (8-bit digits from the highest differing bit) and those are ranked.
__device__ int select_block(const uint64_t (&key)[kSelKpt], int k, SelShared& sh) {
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    // ---- valid count (wave ballots) ----
    uint32_t wc = 0;
#pragma unroll
    for (int i = 0; i < kSelKpt; ++i) wc += __popcll(__ballot(key[i] != 0));
    if (lane == 0) sh.wcnt[wave] = wc;
    for (int g = t; g < IS_MAX_K; g += kSelThreads) sh.group[g] = 0;
    __syncthreads();
    uint32_t valid_total = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) valid_total += sh.wcnt[w];
    const int want = (int)min_i64(k, valid_total);

    // ---- 1. lower bound tau ----
    uint64_t tau = 1;  // every valid key is >= 1
    if (want < (int)valid_total) {
        uint64_t tmax = 0;
#pragma unroll
        for (int i = 0; i < kSelKpt; ++i) tmax = key[i] > tmax ? key[i] : tmax;
        if (tmax) atomicMax((unsigned long long*)&sh.group[t % want], (unsigned long long)tmax);
        __syncthreads();
        if (wave == 0) {
            uint64_t mn = ~0ull;
            for (int g = lane; g < want; g += kWave) mn = min(mn, sh.group[g]);
            mn = wave_min64(mn);
            if (lane == 0) sh.tau = mn == 0 ? 1 : mn;  // an empty group: no filtering
        }
        __syncthreads();
        tau = sh.tau;
    }

    // ---- 2. candidates: keys >= tau, compacted by wave ballots ----
    uint64_t mask[kSelKpt];
    wc = 0;
#pragma unroll
    for (int i = 0; i < kSelKpt; ++i) {
        mask[i] = __ballot(key[i] >= tau);
        wc += __popcll(mask[i]);
    }
    __syncthreads();  // wcnt reuse
    if (lane == 0) sh.wcnt[wave] = wc;
    __syncthreads();
    uint32_t cand_total = 0, woff = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
        const uint32_t c = sh.wcnt[w];
        woff += w < wave ? c : 0;
        cand_total += c;
    }
    if (cand_total <= (uint32_t)kSelRankMax) {
        uint32_t at = woff;
#pragma unroll
        for (int i = 0; i < kSelKpt; ++i) {
            if (key[i] >= tau) sh.cand[at + lanes_below(mask[i])] = key[i];
            at += __popcll(mask[i]);
        }
        __syncthreads();
        rank_candidates(cand_total, want, sh);
    } else {
        // many candidates: radix select the `want` largest among them
        uint64_t ref = 0, diff = 0;
#pragma unroll
        for (int i = 0; i < kSelKpt; ++i) ref = key[i] >= tau && key[i] > ref ? key[i] : ref;
        if (t == 0) sh.tau = 0;
        __syncthreads();
        if (ref) atomicMax((unsigned long long*)&sh.tau, (unsigned long long)ref);
        __syncthreads();
        ref = sh.tau;  // the largest candidate
#pragma unroll
        for (int i = 0; i < kSelKpt; ++i)
            if (key[i] >= tau) diff |= key[i] ^ ref;
        diff = wave_or64(diff);
        __syncthreads();
        if (lane == 0) sh.group[wave] = diff;
        __syncthreads();
        diff = 0;
#pragma unroll
        for (int w = 0; w < kSelWaves; ++w) diff |= sh.group[w];
        int hi = 63 - __builtin_clzll(diff | 1ull);
        uint64_t pmask = hi == 63 ? 0ull : ~((1ull << (hi + 1)) - 1);
        uint64_t prefix = ref & pmask;
        uint32_t remaining = (uint32_t)want;
        while (true) {
            const int lo = max(0, hi - 7);
            const int width = hi - lo + 1;
            const uint32_t dmask = (1u << width) - 1u;
            if (t < 256) sh.hist[t] = 0;
            __syncthreads();
#pragma unroll
            for (int i = 0; i < kSelKpt; ++i)
                if (key[i] >= tau && (key[i] & pmask) == prefix)
                    atomicAdd(&sh.hist[(uint32_t)(key[i] >> lo) & dmask], 1u);
            __syncthreads();
            if (wave == 0) {
                // suffix sums over the 256 bins: lane L owns bins 4L..4L+3
                const uint32_t b0 = sh.hist[4 * lane], b1 = sh.hist[4 * lane + 1];
                const uint32_t b2 = sh.hist[4 * lane + 2], b3 = sh.hist[4 * lane + 3];
                const uint32_t mine = b0 + b1 + b2 + b3;
                uint32_t incl = mine;  // sum over lanes >= lane
#pragma unroll
                for (int off = 1; off < 64; off <<= 1) {
                    const uint32_t o = __shfl_down(incl, off, kWave);
                    if (lane + off < 64) incl += o;
                }
                const uint32_t a3 = incl - mine, a2 = a3 + b3, a1 = a2 + b2, a0 = a1 + b1;
                if (a3 < remaining && remaining <= a3 + b3) { sh.digit = 4 * lane + 3; sh.above = a3; }
                if (a2 < remaining && remaining <= a2 + b2) { sh.digit = 4 * lane + 2; sh.above = a2; }
                if (a1 < remaining && remaining <= a1 + b1) { sh.digit = 4 * lane + 1; sh.above = a1; }
                if (a0 < remaining && remaining <= a0 + b0) { sh.digit = 4 * lane; sh.above = a0; }
            }
            __syncthreads();
            const uint32_t dg = sh.digit;
            remaining -= sh.above;
            const uint32_t inbin = sh.hist[dg];
            prefix |= (uint64_t)dg << lo;
            pmask |= (uint64_t)dmask << lo;
            __syncthreads();  // hist is rewritten by the next pass
            if (inbin == remaining || lo == 0) break;
            hi = lo - 1;
        }
        // the `want` winners, then their ranks among themselves
        if (t == 0) sh.count = 0;
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kSelKpt; ++i)
            if (key[i] >= tau && (key[i] & pmask) >= prefix) {
                const uint32_t pos = atomicAdd(&sh.count, 1u);
                if (pos < (uint32_t)want) sh.cand[pos] = key[i];
            }
        __syncthreads();
        for (int c = t; c < want; c += kSelThreads) {
            const uint64_t me = sh.cand[c];
            int rank = 0;
            for (int j = 0; j < want; ++j) rank += sh.cand[j] > me;
            sh.sel[rank] = me;
        }
        __syncthreads();
    }

    return want;
}

// Top-k of one chunk of up to kSelThreads * kSelKpt keys per block (keys
// [nq][M], 0 marks an empty entry). With out_ids the block writes the final
// ranking, else its `k` winners (0-padded) to cand_out[q][chunk][k].
__global__ __launch_bounds__(kSelThreads) void select_kernel(const uint64_t* __restrict__ keys_in,
                                                             int64_t M, int k, int nchunks,
                                                             uint64_t* __restrict__ cand_out,
                                                             int32_t* __restrict__ out_ids,
                                                             float* __restrict__ out_scores) {
    __shared__ SelShared sh;
    const int t = threadIdx.x;
    const int q = blockIdx.y;
    const int64_t c0 = (int64_t)blockIdx.x * (kSelThreads * kSelKpt);

    // every load is issued before the first is used: an index past the end
    // re-reads the last key (M >= 1), which is then dropped
    uint64_t key[kSelKpt];
#pragma unroll
    for (int i = 0; i < kSelKpt; ++i) {
        const int64_t idx = c0 + t + (int64_t)i * kSelThreads;  // coalesced
        key[i] = keys_in[(int64_t)q * M + (idx < M ? idx : M - 1)];
    }
#pragma unroll
    for (int i = 0; i < kSelKpt; ++i) {
        const int64_t idx = c0 + t + (int64_t)i * kSelThreads;
        key[i] = idx < M ? key[i] : 0ull;
    }
    // key[i] is nonzero iff valid: ~id has its top bit set for ids < 2^31
    const int want = select_block(key, k, sh);

    // ---- output, best first ----
    if (out_ids) {
        for (int i = t; i < want; i += kSelThreads) {
            const uint64_t me = sh.sel[i];
            out_ids[(int64_t)q * k + i] = (int32_t)key_id(me);
            if (out_scores) out_scores[(int64_t)q * k + i] = key_score(me);
        }
    } else {
        uint64_t* dst = cand_out + ((int64_t)q * nchunks + blockIdx.x) * k;
        for (int i = t; i < k; i += kSelThreads) dst[i] = i < want ? sh.sel[i] : 0ull;
    }
}

// Largest / smallest value over the 64 lanes of a wave (uniform result): DPP
// quad, half-row and row exchanges give every lane its 16-lane row's value,
// the four rows are combined in scalar registers.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));
    const uint32_t r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
    const uint32_t r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
    return max(max(r0, r1), max(r2, r3));
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));
    const uint32_t r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
    const uint32_t r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
    return min(min(r0, r1), min(r2, r3));
}

// Final top-k of at most kSelThreads * KPT fp32 scores per query, one block
// per query (the single-chunk case: one query against a bank of up to 16,384
// facts). One CU does all of it, so the work per key is kept small:
//  * thresholds are taken on the 32-bit order-preserving images of the
//    scores (the id only breaks ties, so it is attached to candidates only);
//  * the lower bound tau is the lower edge of a narrow bin holding the
//    want-th largest thread maximum: radix passes of 8 bits over the thread
//    maxima, from the highest bit where they differ, until at most 32 of them
//    share the bin; at least `want` scores are >= tau and typically few more;
//  * the candidates (valid, score bits >= tau) get their 64-bit rank keys,
//    are gathered in LDS (each wave reserves its run with one atomic) and
//    ranked pairwise. Should there be more than kSelRankMax of them (many
//    tied scores), the general select over 64-bit keys takes over.
//
// With cand_out the block ranks chunk blockIdx.x (kSelThreads * KPT scores
// from index blockIdx.x * kSelThreads * KPT of the query's row of Mrow) and
// writes its k winners as keys, best first and 0-padded, to
// cand_out[q][chunk][k]; otherwise the row (M = Mrow scores) is one chunk
// and the ranking goes to out_ids / out_scores.
template <int KPT>
__global__ __launch_bounds__(kSelThreads) void select_small_kernel(
    const float* __restrict__ scores, int64_t Mrow, int k, int32_t* __restrict__ out_ids,
    float* __restrict__ out_scores, uint64_t* __restrict__ cand_out, int nchunks) {
    __shared__ SelShared sh;
    __shared__ uint32_t s_hist2[256];   // radix passes alternate between sh.hist and this
    __shared__ uint32_t s_ncand;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int q = blockIdx.y;
    const int64_t base = cand_out ? (int64_t)blockIdx.x * (kSelThreads * KPT) : 0;
    const int64_t M = cand_out ? min_i64(Mrow - base, (int64_t)kSelThreads * KPT) : Mrow;
    const float* sq = scores + (int64_t)q * Mrow + base;
    // all loads issued before the first is used (an index past the end
    // re-reads the last score, M >= 1, and is then dropped)
    float sv[KPT];
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
        const int64_t idx = t + (int64_t)i * kSelThreads;  // coalesced
        sv[i] = sq[idx < M ? idx : M - 1];
    }
    uint32_t u[KPT];
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
        const int64_t idx = t + (int64_t)i * kSelThreads;
        u[i] = idx < M ? score_order_bits(sv[i]) : 0u;
    }
    const int want = (int)min_i64(k, M);
    // the thread's keys are valid for i < nv (NaN scores are valid, lowest)
    const int nv = M > t ? (int)min_i64(KPT, (M - t + kSelThreads - 1) / kSelThreads) : 0;
    if (t == 0) s_ncand = 0;

    // ---- 1. lower bound tau on the score bits ----
    uint32_t tau = 0;  // every valid key is a candidate
    if ((int64_t)want < M) {
        uint32_t tm = 0;
#pragma unroll
        for (int i = 0; i < KPT; ++i) tm = (i < nv && u[i] > tm) ? u[i] : tm;
        // holders: the min(M, kSelThreads) >= want threads with a valid key.
        // Maxima of non-negative scores (top bit set) are bracketed on their
        // own when there are at least `want` of them, so that a single
        // negative maximum does not widen the first radix window to the sign
        const bool nonneg = nv > 0 && (tm & 0x80000000u) != 0;
        const uint32_t wmax = wave_max_u32(tm);
        const uint32_t wmin = wave_min_u32(nv > 0 ? tm : 0xFFFFFFFFu);
        const uint32_t wmin_nn = wave_min_u32(nonneg ? tm : 0xFFFFFFFFu);
        const uint32_t wnn = (uint32_t)__popcll(__ballot(nonneg));
        if (lane == 0) {
            sh.group[wave] = wmax;
            sh.group[kSelWaves + wave] = wmin;
            sh.group[2 * kSelWaves + wave] = wmin_nn;
            sh.group[3 * kSelWaves + wave] = wnn;
        }
        if (t < 256) {
            sh.hist[t] = 0;
            s_hist2[t] = 0;
        }
        __syncthreads();
        // every wave combines the 16 waves' statistics itself: lane l reads
        // entry l of the four 16-entry tables and each 16-lane row reduces its
        // table (max, min, min, sum) with exchanges inside the row (one LDS
        // read per lane instead of 64)
        static_assert(4 * kSelWaves == kWave, "four tables of one entry per wave");
        const int row = lane >> 4;
        uint32_t gv = (uint32_t)sh.group[lane];
#pragma unroll
        for (int off = 8; off >= 1; off >>= 1) {
            const uint32_t o = __shfl_xor(gv, off, kWave);
            gv = row == 0 ? max(gv, o) : (row == 3 ? gv + o : min(gv, o));
        }
        const uint32_t ref = __builtin_amdgcn_readlane(gv, 0);
        uint32_t lowest = __builtin_amdgcn_readlane(gv, 16);
        const uint32_t lowest_nn = __builtin_amdgcn_readlane(gv, 32);
        const uint32_t n_nn = __builtin_amdgcn_readlane(gv, 48);
        if (n_nn >= (uint32_t)want) lowest = lowest_nn;
        // at least `want` maxima lie in [lowest, ref]; those below are left
        // out of the histogram by the prefix test
        const uint32_t diff = ref ^ lowest;
        if (diff == 0) {
            tau = ref;
        } else {
            int hi = 31 - __builtin_clz(diff);
            uint32_t pmask = hi == 31 ? 0u : ~((1u << (hi + 1)) - 1u);
            uint32_t prefix = ref & pmask;
            uint32_t need = (uint32_t)want;
            for (int pass = 0;; ++pass) {
                uint32_t* hist = (pass & 1) ? s_hist2 : sh.hist;
                const int lo = max(0, hi - 7);
                const uint32_t dmask = (1u << (hi - lo + 1)) - 1u;
                if (nv > 0 && (tm & pmask) == prefix) atomicAdd(&hist[(tm >> lo) & dmask], 1u);
                __syncthreads();
                if (wave == 0) {
                    // suffix sums over the bins (lane L owns bins 4L..4L+3); the
                    // bin where the count of maxima from the top reaches `need`
                    const uint32_t b0 = hist[4 * lane], b1 = hist[4 * lane + 1];
                    const uint32_t b2 = hist[4 * lane + 2], b3 = hist[4 * lane + 3];
                    const uint32_t mine = b0 + b1 + b2 + b3;
                    uint32_t incl = mine;  // sum over lanes >= lane
#pragma unroll
                    for (int off = 1; off < 64; off <<= 1) {
                        const uint32_t o = __shfl_down(incl, off, kWave);
                        if (lane + off < 64) incl += o;
                    }
                    const uint32_t a3 = incl - mine, a2 = a3 + b3, a1 = a2 + b2, a0 = a1 + b1;
                    if (a3 < need && need <= a3 + b3) { sh.digit = 4 * lane + 3; sh.above = a3; sh.count = b3; }
                    if (a2 < need && need <= a2 + b2) { sh.digit = 4 * lane + 2; sh.above = a2; sh.count = b2; }
                    if (a1 < need && need <= a1 + b1) { sh.digit = 4 * lane + 1; sh.above = a1; sh.count = b1; }
                    if (a0 < need && need <= a0 + b0) { sh.digit = 4 * lane; sh.above = a0; sh.count = b0; }
                }
                __syncthreads();
                const uint32_t inbin = sh.count;
                prefix |= sh.digit << lo;
                pmask |= dmask << lo;
                need -= sh.above;
                // this pass's bins are cleared for the pass after next; the next
                // pass's barrier orders the clearing before that pass's counts
                // and wave 0's rewrite of digit / above / count after the reads
                if (t < 256) hist[t] = 0;
                if (inbin <= 32u || lo == 0) break;
                hi = lo - 1;
            }
            tau = prefix;  // the lower edge of the bin: >= want maxima are >= tau
        }
    } else {
        __syncthreads();  // s_ncand is cleared before any wave counts into it
    }

    // ---- 2. candidates: valid keys with score bits >= tau ----
    uint64_t mask[KPT];
    uint32_t wc = 0;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
        mask[i] = __ballot(i < nv && u[i] >= tau);
        wc += __popcll(mask[i]);
    }
    uint32_t at = 0;
    if (lane == 0 && wc) at = atomicAdd(&s_ncand, wc);
    at = __shfl(at, 0, kWave);
    if (wc) {
#pragma unroll
        for (int i = 0; i < KPT; ++i) {
            if (mask[i]) {  // wave-uniform: most of the masks are empty
                if (u[i] >= tau && i < nv) {
                    const uint32_t idx = (uint32_t)(base + t + i * kSelThreads);
                    const uint32_t slot = at + lanes_below(mask[i]);
                    if (slot < (uint32_t)kSelRankMax)
                        sh.cand[slot] = ((uint64_t)u[i] << 32) | (uint64_t)(~idx);
                }
                at += __popcll(mask[i]);
            }
        }
    }
    __syncthreads();
    const uint32_t cand_total = s_ncand;
    int got = want;
    if (cand_total <= (uint32_t)kSelRankMax) {
        rank_candidates(cand_total, want, sh);
    } else {
        uint64_t key[kSelKpt];
#pragma unroll
        for (int i = 0; i < kSelKpt; ++i) {
            const uint32_t idx = (uint32_t)(base + t + i * kSelThreads);
            key[i] = (i < KPT && i < nv) ? (((uint64_t)u[i] << 32) | (uint64_t)(~idx)) : 0ull;
        }
        got = select_block(key, k, sh);
    }

    // ---- output, best first ----
    if (cand_out) {
        uint64_t* dst = cand_out + ((int64_t)q * nchunks + blockIdx.x) * k;
        for (int i = t; i < k; i += kSelThreads) dst[i] = i < got ? sh.sel[i] : 0ull;
        return;
    }
    for (int i = t; i < got; i += kSelThreads) {
        const uint64_t me = sh.sel[i];
        out_ids[(int64_t)q * k + i] = (int32_t)key_id(me);
        if (out_scores) out_scores[(int64_t)q * k + i] = key_score(me);
    }
}

// Final ranking of per-chunk winner lists: nlists lists of k keys per query,
// each best first and 0-padded, all keys distinct. A key's rank is its
// position in its own list plus, in every other list, the number of keys
// above it (a binary search), so one pass over the lists in shared memory
// ranks them all; the keys ranked below k are the answer.
constexpr int kMergeMax = 4096;  // keys per query at most

__global__ __launch_bounds__(kSelThreads) void merge_ranked_kernel(
    const uint64_t* __restrict__ lists, int nlists, int k, int32_t* __restrict__ out_ids,
    float* __restrict__ out_scores, uint64_t* __restrict__ out_keys) {
    __shared__ uint64_t s[kMergeMax];
    const int q = blockIdx.x;
    const int total = nlists * k;
    const uint64_t* src = lists + (int64_t)q * total;
    for (int e = threadIdx.x; e < total; e += kSelThreads) s[e] = src[e];
    // key output: every position starts empty (the barrier orders these
    // writes before the ranked ones)
    if (out_keys)
        for (int i = threadIdx.x; i < k; i += kSelThreads) out_keys[(int64_t)q * k + i] = 0ull;
    __syncthreads();
    for (int e = threadIdx.x; e < total; e += kSelThreads) {
        const uint64_t x = s[e];
        if (x == 0) continue;  // padding
        const int c = e / k;
        int rank = e - c * k;
        for (int c2 = 0; c2 < nlists; ++c2) {
            if (c2 == c) continue;
            const uint64_t* l = s + c2 * k;
            int lo = 0, hi = k;  // first position whose key is below x
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (l[mid] > x) lo = mid + 1;
                else hi = mid;
            }
            rank += lo;
        }
        if (rank < k) {
            if (out_keys) {
                out_keys[(int64_t)q * k + rank] = x;
            } else {
                out_ids[(int64_t)q * k + rank] = (int32_t)key_id(x);
                if (out_scores) out_scores[(int64_t)q * k + rank] = key_score(x);
            }
        }
    }
}

// Final ranking of the filtered matrix-core scan, one block per query. The
// candidates of query q are the k keys of the sample, `first[q][0 .. k)`,
// then the survivors of every scan block g, regions[q][g][0 .. counts[q][g]).
// They are taken in chunks: the first chunk holds the first
// kSelThreads * kSelKpt candidates; every later chunk holds the winners so
// far and the next candidates, so any number of survivors is ranked exactly.
__global__ __launch_bounds__(kSelThreads) void select_regions_kernel(
    const uint64_t* __restrict__ first, const uint64_t* __restrict__ regions,
    const uint32_t* __restrict__ counts, int G, int64_t rcap, int k,
    int32_t* __restrict__ out_ids, float* __restrict__ out_scores) {
    __shared__ SelShared sh;
    __shared__ int64_t s_pre[kSelThreads + 1];   // survivors before region g
    __shared__ int64_t s_wave_tot[kSelWaves];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int q = blockIdx.x;
    const uint64_t* fq = first + (int64_t)q * k;
    const uint64_t* rq = regions + (int64_t)q * G * rcap;

    // exclusive prefix of the region counts (G <= kSelThreads)
    const int64_t c = t < G ? (int64_t)counts[(int64_t)q * G + t] : 0;
    const int64_t incl = wave_incl_scan(c, lane);
    if (lane == 63) s_wave_tot[wave] = incl;
    __syncthreads();
    int64_t excl = incl - c;
    for (int w = 0; w < wave; ++w) excl += s_wave_tot[w];
    if (t < G) s_pre[t] = excl;
    if (t == G - 1) s_pre[G] = excl + c;  // all survivors
    __syncthreads();
    const int64_t total = (int64_t)k + s_pre[G];

    constexpr int64_t kChunk = (int64_t)kSelThreads * kSelKpt;
    int64_t next = 0;   // candidates consumed so far
    int carried = 0;    // winners carried into this chunk (slots 0 .. carried)
    uint64_t carry = 0;
    int want;
    while (true) {
        // every slot's candidate is loaded before any is used (a slot without
        // one re-reads fq[0], k >= 1, and drops it): loads under per-slot
        // conditions are compiled into branches that each wait for their load
        uint64_t key[kSelKpt];
        uint32_t have = 0;  // bit i: slot i holds a candidate
#pragma unroll
        for (int i = 0; i < kSelKpt; ++i) {
            const int64_t slot = t + (int64_t)i * kSelThreads;
            const int64_t x = next + slot - carried;
            const uint64_t* src = fq;
            if (slot >= carried && x < total) {
                have |= 1u << i;
                if (x < k) {
                    src = fq + x;
                } else {
                    const int64_t y = x - k;
                    int lo = 0, hi = G - 1;  // last region g with s_pre[g] <= y
                    while (lo < hi) {
                        const int mid = (lo + hi + 1) >> 1;
                        if (s_pre[mid] <= y) lo = mid; else hi = mid - 1;
                    }
                    src = rq + (int64_t)lo * rcap + (y - s_pre[lo]);
                }
            }
            key[i] = *src;
        }
#pragma unroll
        for (int i = 0; i < kSelKpt; ++i) {
            const int64_t slot = t + (int64_t)i * kSelThreads;
            // a carried winner (only i == 0 and t < carried), a candidate, or empty
            key[i] = slot < carried ? carry : ((have >> i) & 1u ? key[i] : 0ull);
        }
        next += kChunk - carried;
        want = select_block(key, k, sh);
        if (next >= total) break;
        carried = want;
        carry = t < want ? sh.sel[t] : 0ull;
        __syncthreads();  // sel is rewritten by the next chunk
    }
    for (int i = t; i < want; i += kSelThreads) {
        const uint64_t me = sh.sel[i];
        out_ids[(int64_t)q * k + i] = (int32_t)key_id(me);
        if (out_scores) out_scores[(int64_t)q * k + i] = key_score(me);
    }
}

int64_t select_chunk_len() { return (int64_t)kSelThreads * kSelKpt; }

hipError_t launch_select_scores(const float* scores, int64_t n, int k, int nq, int nchunks,
                                uint64_t* cand, hipStream_t st) {
    dim3 grid((unsigned)nchunks, (unsigned)nq);
    hipLaunchKernelGGL((select_small_kernel<kSelKpt>), grid, dim3(kSelThreads), 0, st, scores, n,
                       k, (int32_t*)nullptr, (float*)nullptr, cand, nchunks);
    return hipGetLastError();
}

bool merge_ranked_applies(int nlists, int k) { return (int64_t)nlists * k <= kMergeMax; }

hipError_t launch_merge_ranked(const uint64_t* lists, int nlists, int k, int nq, int32_t* out_ids,
                               float* out_scores, uint64_t* out_keys, hipStream_t st) {
    if (!merge_ranked_applies(nlists, k)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(merge_ranked_kernel, dim3((unsigned)nq), dim3(kSelThreads), 0, st, lists,
                       nlists, k, out_ids, out_scores, out_keys);
    return hipGetLastError();
}

hipError_t launch_select_small(const float* scores, int64_t n, int k, int nq, int32_t* out_ids,
                               float* out_scores, hipStream_t st) {
    const int64_t kpt = (n + kSelThreads - 1) / kSelThreads;
    dim3 grid(1u, (unsigned)nq);
#define IS_SELECT_SMALL(KPT)                                                                      \
    hipLaunchKernelGGL((select_small_kernel<KPT>), grid, dim3(kSelThreads), 0, st, scores, n, k,  \
                       out_ids, out_scores, (uint64_t*)nullptr, 1)
    if (kpt <= 4) IS_SELECT_SMALL(4);
    else if (kpt <= 8) IS_SELECT_SMALL(8);
    else if (kpt <= 12) IS_SELECT_SMALL(12);
    else if (kpt <= 16) IS_SELECT_SMALL(16);
    else return hipErrorInvalidValue;
#undef IS_SELECT_SMALL
    return hipGetLastError();
}

hipError_t launch_select_keys(const uint64_t* keys, int64_t M, int k, int nq, int nchunks,
                              uint64_t* cand, int32_t* out_ids, float* out_scores, hipStream_t st) {
    dim3 grid((unsigned)nchunks, (unsigned)nq);
    hipLaunchKernelGGL(select_kernel, grid, dim3(kSelThreads), 0, st, keys, M, k, nchunks, cand,
                       out_ids, out_scores);
    return hipGetLastError();
}

hipError_t launch_select_regions(const uint64_t* first, const uint64_t* regions,
                                 const uint32_t* counts, int G, int64_t rcap, int k, int nq,
                                 int32_t* out_ids, float* out_scores, hipStream_t st) {
    if (G < 1 || G > kSelThreads) return hipErrorInvalidValue;
    hipLaunchKernelGGL(select_regions_kernel, dim3((unsigned)nq), dim3(kSelThreads), 0, st, first,
                       regions, counts, G, rcap, k, out_ids, out_scores);
    return hipGetLastError();
}

}  // namespace is
