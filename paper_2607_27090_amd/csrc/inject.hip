// Fused gather + Chunked-RoPE + scatter into the paged KV cache (§3.3
// composition: stored pre-RoPE keys are rotated on the fly to the positions
// the request assigns; §3.4: the composed K and V go into the request's
// blocks through the slot mapping; §2.4 / Theorem "Chunked RoPE Injection",
// §5.1: R_p is the block-diagonal rotation by p * theta^(-2j/D), or by p
// times the model's own rotary table, §3.3 and §6.1).
//
// Work decomposition (HBM-bound streaming copy with a little math):
//   * a lane item is (placed token, 16-element lane unit of a head): the lane
//     owns elements [8u, 8u+8) of the first half of head h and the matching
//     elements [D/2 + 8u, D/2 + 8u + 8) of the second half, so every rotation
//     pair lives in one lane in both pair layouts -- (j, j + D/2), the
//     half-split one, and (2j, 2j + 1), the interleaved one -- and all
//     loads/stores are 16 bytes; one wave covers 64 consecutive lane items,
//     i.e. one full (token, layer) row of H*D elements when H*D == 1024
//     (2 KiB of K and 2 KiB of V, read and written as whole 128-byte lines);
//   * a work item is (64 consecutive lane items, kInjLayers consecutive
//     layers), numbered layer-group major; a request's work items are dealt
//     round robin to its workgroups, so all CUs sweep the request together
//     (HBM serves one front of neighbouring addresses better than one
//     contiguous share per CU: a plain copy of 526 MB runs at 5.6 TB/s in
//     grid-stride order and at 4.5 TB/s with a contiguous share per CU), in
//     an XCD-aware order: neighbouring items go to the workgroups of one XCD;
//   * a workgroup is 12 waves and occupies a whole CU (the launch reserves
//     more than half of the CU's LDS), and its waves take the workgroup's
//     work items one at a time from a counter in LDS. The hardware issues the
//     memory instructions of older waves first, so waves of one CU progress
//     at very different rates; taking items from a shared counter lets the
//     favoured waves do more of them, where equal static shares per wave or
//     per co-resident workgroup left the least favoured finishing last;
//   * each item's 8 angles per lane (fp64 reduction + fp32 sincos) are
//     computed while its loads are in flight;
//   * loads and stores are non-temporal: every stored byte is read once and
//     every page byte is written once.
//
// The same kernel with PLACE set also does the placement and slot mapping
// (§5.2 position policy, §2.2 block tables) itself: its set-up already
// forms the placement offsets b_i, so a token's position is start_pos + idx
// and its slot comes from the block table, the request is validated exactly
// as the slot map validates it, and the slots, positions and m are written
// as by-products. This saves the slot map's own launch on the request's
// critical path.
#include <atomic>

#include "common.hpp"
#include "launch.hpp"

namespace is {

// 12 waves, three per SIMD: one workgroup fills a CU. More waves in flight
// serve this scattered pattern worse (1,024 threads were 1.8% slower, 512
// threads 10% slower than 768)
constexpr int kInjThreads = 768;
constexpr int kInjFacts = 2;       // consecutive facts of the placement per thread in set-up
constexpr int kInjLayers = 1;      // layers of one work item (2 and 4 measured slower)
// block-table entries each thread loads with the fact ids (PLACE); blocks
// beyond 2 * 1024 are read after the scan
constexpr int kInjBtAhead = 2;

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// 16-byte non-temporal load / store (streamed: read once, written once)
__device__ __forceinline__ uint4 load_nt(const uint4* p) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void store_nt(uint4* p, uint4 v) {
    const u32x4_t x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<u32x4_t*>(p));
}

__device__ __forceinline__ void rotate8(const uint4 lo, const uint4 hi, const float (&c)[8],
                                        const float (&s)[8], uint4& out_lo, uint4& out_hi) {
    const uint32_t a[4] = {lo.x, lo.y, lo.z, lo.w};
    const uint32_t b[4] = {hi.x, hi.y, hi.z, hi.w};
    uint32_t ya[4], yb[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const float x0a = bf16_lo(a[w]), x0b = bf16_hi(a[w]);  // elements 2w, 2w+1 (first half)
        const float x1a = bf16_lo(b[w]), x1b = bf16_hi(b[w]);  // their partners (second half)
        const int e0 = 2 * w, e1 = 2 * w + 1;
        const float y0a = fmaf(x0a, c[e0], -(x1a * s[e0]));
        const float y1a = fmaf(x1a, c[e0], x0a * s[e0]);
        const float y0b = fmaf(x0b, c[e1], -(x1b * s[e1]));
        const float y1b = fmaf(x1b, c[e1], x0b * s[e1]);
        ya[w] = pack_bf16x2(y0a, y0b);
        yb[w] = pack_bf16x2(y1a, y1b);
    }
    out_lo = make_uint4(ya[0], ya[1], ya[2], ya[3]);
    out_hi = make_uint4(yb[0], yb[1], yb[2], yb[3]);
}

// Interleaved layout: every 32-bit word of lo / hi is one pair (2j, 2j + 1);
// lo holds pairs with angles c[0..3] / s[0..3], hi those with c[4..7] / s[4..7].
__device__ __forceinline__ void rotate8_interleaved(const uint4 lo, const uint4 hi,
                                                    const float (&c)[8], const float (&s)[8],
                                                    uint4& out_lo, uint4& out_hi) {
    const uint32_t in[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    uint32_t out[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float x0 = bf16_lo(in[e]), x1 = bf16_hi(in[e]);
        const float y0 = fmaf(x0, c[e], -(x1 * s[e]));
        const float y1 = fmaf(x1, c[e], x0 * s[e]);
        out[e] = pack_bf16x2(y0, y1);
    }
    out_lo = make_uint4(out[0], out[1], out[2], out[3]);
    out_hi = make_uint4(out[4], out[5], out[6], out[7]);
}

// PLACE = false: slots, positions and m_dev are the slot map's outputs.
// PLACE = true: they are not read; pl holds the block table and the outputs.
template <bool INTERLEAVED, bool PLACE>
__global__ __launch_bounds__(kInjThreads, 1) void inject_kernel(
    const int32_t* __restrict__ ids, const uint4* __restrict__ preK, const uint4* __restrict__ V,
    const int64_t* __restrict__ slots, const int32_t* __restrict__ positions, float rope_theta,
    uint4* __restrict__ paged_k, uint4* __restrict__ paged_v,
    const int64_t* __restrict__ fact_offsets, const int32_t* __restrict__ fact_lens,
    const int32_t* __restrict__ m_dev, int32_t k, int64_t n, int64_t lens_stride,
    int32_t reverse_rank, int32_t max_tokens, int32_t L, int32_t H, int32_t D, int64_t T_store,
    int64_t num_slots, const double* __restrict__ inv_freq, uint32_t* __restrict__ status,
    PlaceArgs pl) {
    __shared__ int64_t s_b[IS_MAX_K + 1];     // placed-token offset of each fact
    __shared__ int64_t s_off[IS_MAX_K];       // store row of each fact, -1: skip
    __shared__ double s_invf[IS_MAX_HEAD_DIM / 2];
    __shared__ int64_t s_wave_tot[kInjThreads / kWave];
    __shared__ uint32_t s_flags;
    __shared__ int32_t s_bad;
    __shared__ int32_t s_bad_block;           // PLACE: a used block-table entry is < 0
    __shared__ int64_t s_first_neg;           // PLACE: lowest preloaded block whose entry is < 0
    __shared__ int32_t s_next;                // next work item of this workgroup

    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int r = blockIdx.y;
    // m and this thread's fact ids (facts kInjFacts * t + f of the placement
    // order) are independent loads; a fact's length and store row depend
    // only on its id and are loaded together
    const int32_t m_in = PLACE ? 0 : m_dev[r];
    const int32_t* rid = ids + (int64_t)r * k;
    int32_t cid[kInjFacts];
#pragma unroll
    for (int f = 0; f < kInjFacts; ++f) {
        const int i = kInjFacts * t + f;
        cid[f] = i < k ? (reverse_rank ? rid[k - 1 - i] : rid[i]) : 0;
    }
    // PLACE: the block-table entries of the blocks the first placed tokens
    // can use are independent of everything else and load now too
    const int32_t* bt_r = PLACE ? pl.block_table + (int64_t)r * pl.max_blocks : nullptr;
    const int64_t blk0 = PLACE ? pl.start_pos / pl.page_size : 0;
    int32_t pb[kInjBtAhead] = {};
    if (PLACE) {
        const int64_t blk_cap =
            max_tokens > 0 ? ((int64_t)pl.start_pos + max_tokens - 1) / pl.page_size : -1;
#pragma unroll
        for (int i = 0; i < kInjBtAhead; ++i) {
            const int64_t b = blk0 + t + (int64_t)i * kInjThreads;
            if (b <= blk_cap && b < pl.max_blocks) pb[i] = bt_r[b];
        }
    }
    int32_t m = min(m_in, max_tokens);
    if (!PLACE && m <= 0) return;

    // ---- per-request setup: placement offsets, store rows, frequencies ----
    const int32_t* lens = fact_lens + (int64_t)r * lens_stride;
    const int64_t* offs = fact_offsets + (int64_t)r * lens_stride;
    uint32_t flags = 0;
    int64_t flen[kInjFacts];
    int64_t len = 0;  // this thread's facts together
    // every fact's length and store row are loaded before any is used (an
    // id out of range reads fact 0, n >= 1, and is then dropped): loads
    // under per-fact conditions are compiled into branches that each wait
    // for their load, one memory round trip per load
    int32_t lraw[kInjFacts];
    int64_t oraw[kInjFacts];
#pragma unroll
    for (int f = 0; f < kInjFacts; ++f) {
        const int64_t c = (cid[f] >= 0 && (int64_t)cid[f] < n) ? cid[f] : 0;
        lraw[f] = lens[c];
        oraw[f] = offs[c];
    }
    // (the empty asm keeps the compiler from sinking a load back into the
    // branch that uses it)
#pragma unroll
    for (int f = 0; f < kInjFacts; ++f) asm volatile("" ::"v"(lraw[f]), "v"(oraw[f]));
#pragma unroll
    for (int f = 0; f < kInjFacts; ++f) {
        const int i = kInjFacts * t + f;
        flen[f] = 0;
        if (i < k) {
            int64_t off = -1;
            if (cid[f] < 0 || (int64_t)cid[f] >= n) {
                flags |= IS_DEV_ID_RANGE;
            } else {
                const int32_t l = lraw[f];
                const int64_t o = oraw[f];
                if (l < 0) {
                    flags |= IS_DEV_BAD_LEN;
                } else {
                    flen[f] = l;
                    if (o < 0 || o + l > T_store) flags |= IS_DEV_SRC_RANGE;
                    else off = o;
                }
            }
            s_off[i] = off;
        }
        len += flen[f];
    }
    if (t == 0) {
        s_flags = 0; s_bad = 0; s_bad_block = 0; s_next = 0;
        s_first_neg = INT64_MAX;
    }
    const int64_t incl = wave_incl_scan(len, lane);
    if (lane == 63) s_wave_tot[wave] = incl;
    if (t < (D >> 1))
        s_invf[t] = inv_freq ? inv_freq[t]
                             : exp2(-(2.0 * (double)t / (double)D) * log2((double)rope_theta));
    __syncthreads();
    if (flags & (IS_DEV_ID_RANGE | IS_DEV_BAD_LEN)) s_bad = 1;
    int64_t excl = incl - len;
    for (int w = 0; w < wave; ++w) excl += s_wave_tot[w];
#pragma unroll
    for (int f = 0; f < kInjFacts; ++f) {
        const int i = kInjFacts * t + f;
        if (i < k) s_b[i] = excl;
        excl += flen[f];
    }
    if (t == 0) {
        int64_t tot = 0;
        for (int w = 0; w < kInjThreads / kWave; ++w) tot += s_wave_tot[w];
        s_b[k] = tot;
    }
    // a request-level failure reports only the id / length flags (a store
    // range flag of the thread's other fact is reported with the items)
    if (flags & (IS_DEV_ID_RANGE | IS_DEV_BAD_LEN))
        atomicOr(&s_flags, flags & (IS_DEV_ID_RANGE | IS_DEV_BAD_LEN));
    if (PLACE) {
        // negative entries among the preloaded blocks; whether the placement
        // reaches them is known once the total is
#pragma unroll
        for (int i = 0; i < kInjBtAhead; ++i)
            if (pb[i] < 0)
                atomicMin((unsigned long long*)&s_first_neg,
                          (unsigned long long)(blk0 + t + (int64_t)i * kInjThreads));
    }
    __syncthreads();
    if (s_bad) {
        // a request with an invalid id or length is skipped as a whole
        if (blockIdx.x == 0 && t == 0) {
            if (PLACE) pl.out_m[r] = 0;
            if (status) atomicOr(status, s_flags);
        }
        return;
    }
    if (PLACE) {
        // the slot map's request checks, in its order: capacity, then a block
        // table too short for the last position, then a negative block among
        // those the placement uses; any of them skips the request (m = 0)
        const int64_t total = s_b[k];
        const int64_t blk_last = ((int64_t)pl.start_pos + total - 1) / pl.page_size;
        uint32_t f = 0;
        if (total > max_tokens) f = IS_DEV_CAPACITY;
        else if (total > 0 && blk_last >= pl.max_blocks) f = IS_DEV_BT_SHORT;
        if (f == 0 && total > 0) {
            if (s_first_neg <= blk_last) f = IS_DEV_BAD_BLOCK;
            const int64_t blk_more = blk0 + (int64_t)kInjBtAhead * kInjThreads;
            if (f == 0 && blk_last >= blk_more) {
                // blocks past the preloaded part: one more pass and barrier
                bool bad = false;
                for (int64_t b = blk_more + t; b <= blk_last; b += kInjThreads)
                    if (bt_r[b] < 0) bad = true;
                if (bad) s_bad_block = 1;
                __syncthreads();
                if (s_bad_block) f = IS_DEV_BAD_BLOCK;
            }
        }
        if (f) {
            if (blockIdx.x == 0 && t == 0) {
                pl.out_m[r] = 0;
                if (status) atomicOr(status, f);
            }
            return;
        }
        if (blockIdx.x == 0 && t == 0) pl.out_m[r] = (int32_t)total;
        m = (int32_t)total;
        if (m <= 0) return;
    }
    if (blockIdx.x != 0) flags = 0;  // fact-level flags are reported once per request

    const int lpu = D >> 4;                         // lane units per head
    const int U = H * lpu;                          // lane units per (token, layer) row
    const int64_t items = (int64_t)m * U;
    // never place more tokens than the facts hold, whatever m says
    const int64_t items_ok = min_i64(items, s_b[k] * U);
    const int64_t ngroups = (items + kWave - 1) / kWave;      // 64-item groups
    const int64_t nlg = (L + kInjLayers - 1) / kInjLayers;     // layer groups
    const int64_t total = ngroups * nlg;
    // this workgroup's items are base, base + G, ... (G = the request's
    // workgroups), so at any moment all CUs work on neighbouring items: one
    // front sweeping the request layer group by layer group. Workgroups are
    // dealt to the 8 XCDs round robin (workgroup b of a request runs on XCD
    // b % 8 when G is a multiple of 8), so base gives each XCD a run of G / 8
    // consecutive items: the page and store rows of neighbouring tokens are
    // then translated in one XCD's L2 TLB instead of in several
    const int64_t G = gridDim.x;
    const int64_t base =
        G % 8 == 0 ? (int64_t)(blockIdx.x / 8) + (G / 8) * (blockIdx.x % 8) : blockIdx.x;
    const int64_t span = (total - base + G - 1) / G;
    const int64_t* slots_r = PLACE ? nullptr : slots + (int64_t)r * max_tokens;
    const int32_t* pos_r = PLACE ? nullptr : positions + (int64_t)r * max_tokens;
    int64_t* out_slots_r = PLACE ? pl.out_slots + (int64_t)r * max_tokens : nullptr;
    int32_t* out_pos_r = PLACE ? pl.out_positions + (int64_t)r * max_tokens : nullptr;

    const int64_t row_units = (int64_t)H * D / 8;  // 16-byte units per (token, layer) row
    const int half_units = D >> 4;                 // 16-byte units in half a head
    const int64_t sstride = T_store * row_units;    // one layer of the store
    const int64_t dstride = num_slots * row_units;  // one layer of the pages

    int32_t j = 0;
    if (lane == 0) j = atomicAdd(&s_next, 1);
    j = __shfl(j, 0, kWave);
    while ((int64_t)j < span) {
        const int64_t wi = base + (int64_t)j * G;
        // the wave's next item is taken now; the LDS round trip hides under
        // this item's loads
        int32_t jn = 0;
        if (lane == 0) jn = atomicAdd(&s_next, 1);
        const int64_t lg = wi / ngroups;
        const int64_t item = (wi - lg * ngroups) * kWave + lane;
        const int l0 = (int)lg * kInjLayers;
        const int nl = min(kInjLayers, L - l0);
        if (item < items_ok) {
            const int32_t token = (int32_t)(item / U);
            const int lu = (int)(item - (int64_t)token * U);
            const int h = lu / lpu;
            const int sub = lu - h * lpu;
            // fact holding this placed token: last i with s_b[i] <= token
            int lo = 0, hi = k - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (s_b[mid] <= token) lo = mid; else hi = mid - 1;
            }
            const int64_t off = s_off[lo];
            // PLACE: position start_pos + idx and slot through the block table
            // (start_pos + max_tokens < 2^31, checked on the host); the first
            // lane unit of each token, in the first layer group, writes the
            // token's slot and position out. The slot is formed after the
            // item's data loads are issued (in both branches), so waiting for
            // the block-table entry never delays them.
            const bool writes_out = PLACE && lg == 0 && lu == 0;
            if (off >= 0) {
                const int64_t src = off + (token - s_b[lo]);
                const int64_t col = (int64_t)h * (D >> 3) + sub;  // 16-byte unit within the row
                const uint4* ksrc = preK + src * row_units + col;
                const uint4* vsrc = V + src * row_units + col;
                // loads are unconditional (a short last layer group re-reads
                // its last layer) so the staging stays in registers
                uint4 klo[kInjLayers], khi[kInjLayers], vlo[kInjLayers], vhi[kInjLayers];
#pragma unroll
                for (int q = 0; q < kInjLayers; ++q) {
                    const int64_t so = (int64_t)(l0 + min(q, nl - 1)) * sstride;
                    klo[q] = load_nt(ksrc + so);
                    khi[q] = load_nt(ksrc + so + half_units);
                    vlo[q] = load_nt(vsrc + so);
                    vhi[q] = load_nt(vsrc + so + half_units);
                }
                int64_t slot;
                int32_t pos;
                if (PLACE) {
                    pos = pl.start_pos + token;
                    const int32_t blk = pos / pl.page_size;
                    slot = (int64_t)bt_r[blk] * pl.page_size + (pos - blk * pl.page_size);
                    if (writes_out) {
                        out_slots_r[token] = slot;
                        out_pos_r[token] = pos;
                    }
                } else {
                    slot = slots_r[token];
                    pos = pos_r[token];
                }
                // the item's angles, computed while its loads are in flight:
                // p * w_j formed in fp64, reduced to [-pi, pi] with a
                // two-constant 2*pi, then fp32 sine and cosine
                float cs[8], sn[8];
                const double p = (double)pos;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    // pair of angle e: half-split, j = 8 sub + e; interleaved,
                    // the 4 pairs of each 16-byte half, j = 4 sub + e and
                    // D/4 + 4 sub + e - 4
                    const int pj = INTERLEAVED ? (e < 4 ? 4 * sub + e : (D >> 2) + 4 * sub + e - 4)
                                               : sub * 8 + e;
                    const double a = p * s_invf[pj];
                    const double nrev = rint(a * 0.15915494309189535);
                    double red = fma(-nrev, 6.283185307179586, a);
                    red = fma(-nrev, 2.4492935982947064e-16, red);
                    sincosf((float)red, &sn[e], &cs[e]);
                }
                if (slot < 0 || slot >= num_slots) {
                    flags |= IS_DEV_SLOT_RANGE;
                } else {
                    uint4* kdst = paged_k + slot * row_units + col;
                    uint4* vdst = paged_v + slot * row_units + col;
#pragma unroll
                    for (int q = 0; q < kInjLayers; ++q) {
                        if (q < nl) {
                            uint4 ylo, yhi;
                            if (INTERLEAVED)
                                rotate8_interleaved(klo[q], khi[q], cs, sn, ylo, yhi);
                            else
                                rotate8(klo[q], khi[q], cs, sn, ylo, yhi);
                            const int64_t dq = (int64_t)(l0 + q) * dstride;
                            store_nt(kdst + dq, ylo);
                            store_nt(kdst + dq + half_units, yhi);
                            store_nt(vdst + dq, vlo[q]);
                            store_nt(vdst + dq + half_units, vhi[q]);
                        }
                    }
                }
            } else if (writes_out) {
                // a fact whose rows are outside the store still gets its
                // tokens' slots and positions, as the slot map gives them
                const int32_t pos = pl.start_pos + token;
                const int32_t blk = pos / pl.page_size;
                out_slots_r[token] = (int64_t)bt_r[blk] * pl.page_size + (pos - blk * pl.page_size);
                out_pos_r[token] = pos;
            }
        }
        j = __shfl(jn, 0, kWave);
    }
    if (flags) atomicOr(&s_flags, flags);
    __syncthreads();
    if (t == 0 && s_flags && status) atomicOr(status, s_flags);
}

hipError_t launch_inject(const int32_t* ids, const void* preK, const void* V, const int64_t* slots,
                         const int32_t* positions, float rope_theta, void* paged_k, void* paged_v,
                         const int64_t* fact_offsets, const int32_t* fact_lens, const int32_t* m,
                         int32_t k, int32_t nq, int64_t n, int64_t lens_stride,
                         int32_t reverse_rank, int32_t max_tokens, int32_t L, int32_t H, int32_t D,
                         int64_t T_store, int64_t num_slots, const double* inv_freq,
                         int32_t interleaved, uint32_t* status, hipStream_t st,
                         const PlaceArgs* place) {
    if (k > kInjFacts * kInjThreads) return hipErrorInvalidValue;
    const int64_t U = (int64_t)H * (D >> 4);
    const int64_t groups_max = ((int64_t)max_tokens * U + kWave - 1) / kWave;
    const int64_t items_max = groups_max * ((L + kInjLayers - 1) / kInjLayers);
    // with nothing to place the plain inject has no work; the fused launch
    // still runs to validate the requests and write m
    if (items_max == 0 && !place) return hipSuccess;
    // one workgroup per CU, shared by the requests; the shape depends on
    // max_tokens only, never on m
    const int cus = compute_units();
    int64_t per_req = cus / nq;
    if (per_req > items_max) per_req = items_max;
    if (per_req < 1) per_req = 1;
    dim3 grid((unsigned)per_req, (unsigned)nq);
    // the dynamic LDS reserve and its attribute, once per device (racing
    // threads compute and set the same values): just enough that the
    // kernel's static and dynamic LDS together exceed half of a CU's (80 KiB
    // of 160 KiB on MI355X), so that no two of its workgroups share a CU and
    // the other half stays free for kernels on other streams
    static std::atomic<int> lds_reserve[64];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const bool cached = dev >= 0 && dev < 64;
    int reserve = cached ? lds_reserve[dev].load(std::memory_order_acquire) : 0;
    if (reserve == 0) {
        int lds_per_cu = 0;
        e = hipDeviceGetAttribute(&lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
                                  dev);
        if (e != hipSuccess) return e;
        const void* fns[4] = {(const void*)inject_kernel<false, false>,
                              (const void*)inject_kernel<true, false>,
                              (const void*)inject_kernel<false, true>,
                              (const void*)inject_kernel<true, true>};
        size_t static_lds = 0;
        for (const void* fn : fns) {
            hipFuncAttributes attr;
            e = hipFuncGetAttributes(&attr, fn);
            if (e != hipSuccess) return e;
            if (attr.sharedSizeBytes > static_lds) static_lds = attr.sharedSizeBytes;
        }
        // total > half, in whole KiB; at least 1 KiB so that the value also
        // marks the device as done
        const int64_t need = (int64_t)lds_per_cu / 2 + 1024 - (int64_t)static_lds;
        reserve = (int)((need < 1024 ? 1024 : need + 1023) / 1024 * 1024);
        for (const void* fn : fns) {
            e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, reserve);
            if (e != hipSuccess) return e;
        }
        if (cached) lds_reserve[dev].store(reserve, std::memory_order_release);
    }
    const PlaceArgs pl = place ? *place : PlaceArgs{};
#define IS_LAUNCH_INJECT(IL, PLACE)                                                                \
    hipLaunchKernelGGL((inject_kernel<IL, PLACE>), grid, dim3(kInjThreads), (size_t)reserve, st, \
                       ids, (const uint4*)preK, (const uint4*)V, slots, positions, rope_theta,     \
                       (uint4*)paged_k, (uint4*)paged_v, fact_offsets, fact_lens, m, k, n,         \
                       lens_stride, reverse_rank, max_tokens, L, H, D, T_store, num_slots,         \
                       inv_freq, status, pl)
    if (place) {
        if (interleaved) IS_LAUNCH_INJECT(true, true);
        else IS_LAUNCH_INJECT(false, true);
    } else {
        if (interleaved) IS_LAUNCH_INJECT(true, false);
        else IS_LAUNCH_INJECT(false, false);
    }
#undef IS_LAUNCH_INJECT
    return hipGetLastError();
}

}  // namespace is
