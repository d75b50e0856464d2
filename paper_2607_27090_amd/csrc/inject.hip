// Fused gather + Chunked-RoPE + scatter into the paged KV cache (§3.3
// composition: stored pre-RoPE keys are rotated on the fly to the positions
// the request assigns; §3.4: the composed K and V go into the request's
// blocks through the slot mapping; §2.4 / Theorem "Chunked RoPE Injection",
// §5.1: R_p is the block-diagonal rotation by p * theta^(-2j/D), or by p
// times the model's own rotary table, §3.3 and §6.1).
//
// Work decomposition (HBM-bound streaming copy with a little math):
//   * a thread item is (placed token, 16-element lane unit of a head): it owns
//     elements [8u, 8u+8) of the first half of head h and the matching
//     elements [D/2 + 8u, D/2 + 8u + 8) of the second half, so every rotation
//     pair lives in one thread in both pair layouts -- (j, j + D/2), the
//     half-split one, and (2j, 2j + 1), the interleaved one -- and all
//     loads/stores are 16 bytes;
//     one wave covers one full (token, layer) row of H*D elements when
//     H*D == 1024, i.e. 2 KiB of K and 2 KiB of V, read and written as whole
//     128-byte lines;
//   * a work unit is (256 consecutive thread items, one layer), ordered token
//     block first; every block of a fixed, persistent grid (~4 per CU, set by
//     max_tokens only) takes one contiguous, equal share of its request's
//     units, reading m from device memory, so a request can be enqueued (or
//     captured in a graph) with no host round trip and no tail imbalance;
//   * the 8 angles of a thread depend only on its token's position, so their
//     fp64 reduction and fp32 sincos are paid once per token block of the
//     share and reused for every layer in it;
//   * layers are processed kUnroll at a time with unconditional loads, so
//     each thread keeps 4 * kUnroll independent 16-byte loads in flight and
//     the staging stays in registers.
#include "common.hpp"
#include "launch.hpp"

namespace is {

constexpr int kInjThreads = 256;
constexpr int kUnroll = 4;

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

template <bool INTERLEAVED>
__global__ __launch_bounds__(kInjThreads, 4) void inject_kernel(
    const int32_t* __restrict__ ids, const uint4* __restrict__ preK, const uint4* __restrict__ V,
    const int64_t* __restrict__ slots, const int32_t* __restrict__ positions, float rope_theta,
    uint4* __restrict__ paged_k, uint4* __restrict__ paged_v,
    const int64_t* __restrict__ fact_offsets, const int32_t* __restrict__ fact_lens,
    const int32_t* __restrict__ m_dev, int32_t k, int64_t n, int64_t lens_stride,
    int32_t reverse_rank, int32_t max_tokens, int32_t L, int32_t H, int32_t D, int64_t T_store,
    int64_t num_slots, const double* __restrict__ inv_freq, uint32_t* __restrict__ status) {
    __shared__ int64_t s_b[IS_MAX_K + 1];     // placed-token offset of each fact
    __shared__ int64_t s_off[IS_MAX_K];       // store row of each fact, -1: skip
    __shared__ double s_invf[IS_MAX_HEAD_DIM / 2];
    __shared__ int64_t s_wave_tot[kInjThreads / kWave];
    __shared__ uint32_t s_flags;
    __shared__ int32_t s_bad;

    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int r = blockIdx.y;
    const int32_t* rid = ids + (int64_t)r * k;
    // issue the independent loads first: m, this thread's (up to 4) fact ids
    // of the placement order, and below the first unit's slot and position
    const int32_t m_in = m_dev[r];
    int32_t cid[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int i = 4 * t + e;
        cid[e] = i < k ? (reverse_rank ? rid[k - 1 - i] : rid[i]) : 0;
    }
    const int32_t m = min(m_in, max_tokens);
    if (m <= 0) return;
    const int lpu = D >> 4;              // lane units per head
    const int U = H * lpu;               // lane units per (token, layer) row

    // Work units are (token block of kInjThreads items, layer), token-block
    // major. Each block takes one contiguous, equal share of the units, so
    // consecutive units usually share a token block and its angles.
    const int64_t items = (int64_t)m * U;
    const int64_t ntb = (items + kInjThreads - 1) / kInjThreads;
    const int64_t total = ntb * L;
    const int64_t u0 = total * blockIdx.x / gridDim.x;
    const int64_t u1 = total * (blockIdx.x + 1) / gridDim.x;
    const int64_t* slots_r = slots + (int64_t)r * max_tokens;
    const int32_t* pos_r = positions + (int64_t)r * max_tokens;
    const int64_t pf_tb = u0 < u1 ? u0 / L : -1;
    int64_t pf_slot = -1;
    int32_t pf_pos = 0;
    if (pf_tb >= 0 && pf_tb * kInjThreads + t < items) {
        const int64_t tok = (pf_tb * kInjThreads + t) / U;
        pf_slot = slots_r[tok];
        pf_pos = pos_r[tok];
    }

    // ---- per-request setup: placement offsets, store rows, frequencies ----
    if (t == 0) { s_flags = 0; s_bad = 0; }
    __syncthreads();
    const int32_t* lens = fact_lens + (int64_t)r * lens_stride;
    const int64_t* offs = fact_offsets + (int64_t)r * lens_stride;
    // each thread owns up to 4 consecutive facts of the placement order
    int32_t my_len[4];
    int64_t run = 0;
    uint32_t flags = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int i = 4 * t + e;
        int32_t len = 0;
        if (i < k) {
            const int32_t c = cid[e];
            int64_t off = -1;
            if (c < 0 || (int64_t)c >= n) {
                flags |= IS_DEV_ID_RANGE;
            } else {
                len = lens[c];
                if (len < 0) {
                    flags |= IS_DEV_BAD_LEN;
                    len = 0;
                } else {
                    off = offs[c];
                    if (off < 0 || off + len > T_store) {
                        flags |= IS_DEV_SRC_RANGE;
                        off = -1;
                    }
                }
            }
            s_off[i] = off;
        }
        my_len[e] = len;
        run += len;
    }
    if (flags & (IS_DEV_ID_RANGE | IS_DEV_BAD_LEN)) s_bad = 1;
    // exclusive scan of per-thread totals
    const int64_t incl = wave_incl_scan(run, lane);
    if (lane == 63) s_wave_tot[wave] = incl;
    if (t < (D >> 1))
        s_invf[t] = inv_freq ? inv_freq[t]
                             : exp2(-(2.0 * (double)t / (double)D) * log2((double)rope_theta));
    __syncthreads();
    int64_t excl = incl - run;
    for (int w = 0; w < wave; ++w) excl += s_wave_tot[w];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int i = 4 * t + e;
        if (i < k) s_b[i] = excl;
        excl += my_len[e];
    }
    if (t == 0) {
        int64_t tot = 0;
        for (int w = 0; w < kInjThreads / kWave; ++w) tot += s_wave_tot[w];
        s_b[k] = tot;
    }
    __syncthreads();
    if (s_bad) {
        // a request with an invalid id or length is skipped as a whole
        if (blockIdx.x == 0 && t == 0 && status) atomicOr(status, flags);
        return;
    }
    if (blockIdx.x != 0) flags = 0;  // fact-level flags are reported once per request
    // never place more tokens than the facts hold, whatever m says
    const int64_t items_ok = min(items, s_b[k] * U);

    const int64_t row_units = (int64_t)H * D / 8;  // 16-byte units per (token, layer) row
    const int half_units = D >> 4;                 // 16-byte units in half a head

    const int64_t sstride = T_store * row_units;    // one layer of the store
    const int64_t dstride = num_slots * row_units;  // one layer of the pages
    // the slot and position of the next segment's token are loaded one
    // segment ahead, so a segment switch does not wait on them
    int64_t nx_slot = pf_slot;
    int32_t nx_pos = pf_pos;
    for (int64_t u = u0; u < u1;) {
        const int64_t tb = u / L;
        const int l0 = (int)(u - tb * L);
        const int l1 = (int)min_i64(L, l0 + (u1 - u));
        u += l1 - l0;
        const int64_t slot_in = nx_slot;
        const int32_t pos_in = nx_pos;
        if (u < u1) {
            const int64_t nitem = (u / L) * kInjThreads + t;
            if (nitem < items_ok) {
                const int64_t ntok = nitem / U;
                nx_slot = slots_r[ntok];
                nx_pos = pos_r[ntok];
            }
        }
        const int64_t item = tb * kInjThreads + t;
        if (item >= items_ok) continue;
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
        if (off < 0) continue;
        const int64_t src = off + (token - s_b[lo]);
        const int64_t slot = slot_in;
        if (slot < 0 || slot >= num_slots) { flags |= IS_DEV_SLOT_RANGE; continue; }

        const int64_t col = (int64_t)h * (D >> 3) + sub;  // 16-byte unit within the row
        const uint4* ksrc = preK + src * row_units + col;
        const uint4* vsrc = V + src * row_units + col;
        uint4* kdst = paged_k + slot * row_units + col;
        uint4* vdst = paged_v + slot * row_units + col;

        float cs[8], sn[8];
        for (int l = l0; l < l1; l += kUnroll) {
            // loads are unconditional (a short tail re-reads its last layer)
            // so the staging arrays stay in registers
            uint4 klo[kUnroll], khi[kUnroll], vlo[kUnroll], vhi[kUnroll];
#pragma unroll
            for (int j = 0; j < kUnroll; ++j) {
                const int64_t lj = min(l + j, l1 - 1);
                klo[j] = ksrc[lj * sstride];
                khi[j] = ksrc[lj * sstride + half_units];
                vlo[j] = vsrc[lj * sstride];
                vhi[j] = vsrc[lj * sstride + half_units];
            }
            if (l == l0) {
                // the segment's angles, computed while its first loads are in
                // flight: p * w_j formed in fp64, reduced to [-pi, pi] with a
                // two-constant 2*pi, then fp32 sine and cosine
                const double p = (double)pos_in;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    // pair of angle e: half-split, j = 8 sub + e; interleaved,
                    // the 4 pairs of each 16-byte half, j = 4 sub + e and
                    // D/4 + 4 sub + e - 4
                    const int j = INTERLEAVED ? (e < 4 ? 4 * sub + e : (D >> 2) + 4 * sub + e - 4)
                                              : sub * 8 + e;
                    const double a = p * s_invf[j];
                    const double nrev = rint(a * 0.15915494309189535);
                    double red = fma(-nrev, 6.283185307179586, a);
                    red = fma(-nrev, 2.4492935982947064e-16, red);
                    sincosf((float)red, &sn[e], &cs[e]);
                }
            }
#pragma unroll
            for (int j = 0; j < kUnroll; ++j) {
                uint4 ylo, yhi;
                if (INTERLEAVED)
                    rotate8_interleaved(klo[j], khi[j], cs, sn, ylo, yhi);
                else
                    rotate8(klo[j], khi[j], cs, sn, ylo, yhi);
                if (l + j < l1) {
                    const int64_t dj = (int64_t)(l + j) * dstride;
                    kdst[dj] = ylo;
                    kdst[dj + half_units] = yhi;
                    vdst[dj] = vlo[j];
                    vdst[dj + half_units] = vhi[j];
                }
            }
        }
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
                         int32_t interleaved, uint32_t* status, hipStream_t st) {
    const int64_t U = (int64_t)H * (D >> 4);
    const int64_t ntb_max = ((int64_t)max_tokens * U + kInjThreads - 1) / kInjThreads;
    if (ntb_max == 0) return hipSuccess;
    // a fixed, persistent grid of ~4 blocks per CU shared by the requests;
    // each block takes an equal share of its request's (token block, layer)
    // units, so the shape depends on max_tokens only, never on m
    const int cus = compute_units();
    int64_t per_req = (4LL * cus + nq - 1) / nq;
    if (per_req > ntb_max * L) per_req = ntb_max * L;
    if (per_req < 1) per_req = 1;
    dim3 grid((unsigned)per_req, (unsigned)nq);
    if (interleaved)
        hipLaunchKernelGGL(inject_kernel<true>, grid, dim3(kInjThreads), 0, st, ids,
                           (const uint4*)preK, (const uint4*)V, slots, positions, rope_theta,
                           (uint4*)paged_k, (uint4*)paged_v, fact_offsets, fact_lens, m, k, n,
                           lens_stride, reverse_rank, max_tokens, L, H, D, T_store, num_slots,
                           inv_freq, status);
    else
        hipLaunchKernelGGL(inject_kernel<false>, grid, dim3(kInjThreads), 0, st, ids,
                           (const uint4*)preK, (const uint4*)V, slots, positions, rope_theta,
                           (uint4*)paged_k, (uint4*)paged_v, fact_offsets, fact_lens, m, k, n,
                           lens_stride, reverse_rank, max_tokens, L, H, D, T_store, num_slots,
                           inv_freq, status);
    return hipGetLastError();
}

}  // namespace is
