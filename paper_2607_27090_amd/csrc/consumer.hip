// The consumer of the injected pages: attention logits of each request's
// query against the keys of its placed tokens, read back through the block
// table (Theorem "Chunked RoPE Injection", §5.1: a key rotated at position p
// scores against a query at position N exactly as the stored key would at
// relative position p - N; §3.3: the query follows the memory). Grouped-query
// heads: query head hq reads KV head hq / (Hq / H).
//
//   * one block per (share of the tokens, request); its queries are rotated to
//     qpos[r] once, into shared memory (fp64-reduced angles, fp32 sine and
//     cosine, as the inject kernel rotates keys);
//   * one wave per placed token at a time: the token's slot is resolved from
//     the block table, its K row (H * D bf16) is read in 16-byte units, each
//     lane forms the partial dot products of its 8 elements with the G query
//     heads of that KV head, and the D / 8 lanes of a head reduce them.
#include "common.hpp"
#include "launch.hpp"

namespace is {

constexpr int kConsThreads = 256;
constexpr int kConsWaves = kConsThreads / kWave;
constexpr int kConsMaxQ = 8192;  // Hq * D rotated query elements in shared memory
constexpr int kConsMaxG = 8;     // query heads per KV head

template <bool INTERLEAVED>
__global__ __launch_bounds__(kConsThreads) void paged_scores_kernel(
    const uint16_t* __restrict__ q, const int32_t* __restrict__ qpos,
    const uint4* __restrict__ paged_k, int32_t layer, const int32_t* __restrict__ block_table,
    int32_t page_size, int32_t start_pos, const int32_t* __restrict__ m_dev,
    float* __restrict__ scores, int32_t Hq, int32_t H, int32_t D, int64_t num_slots,
    int32_t max_blocks, int32_t max_tokens, float rope_theta, const double* __restrict__ inv_freq,
    uint32_t* __restrict__ status) {
    __shared__ float s_q[kConsMaxQ];
    __shared__ double s_invf[IS_MAX_HEAD_DIM / 2];
    __shared__ uint32_t s_flags;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int r = blockIdx.y;
    const int half = D >> 1;
    const int m = min(m_dev[r], max_tokens);
    if (t == 0) s_flags = 0;
    if (t < half)
        s_invf[t] = inv_freq ? inv_freq[t]
                             : exp2(-(2.0 * (double)t / (double)D) * log2((double)rope_theta));
    __syncthreads();
    if (m <= 0) return;

    // the query heads, rotated to the query's position
    const double p = (double)qpos[r];
    const uint16_t* qr = q + (int64_t)r * Hq * D;
    for (int i = t; i < Hq * half; i += kConsThreads) {
        const int hq = i / half, j = i - hq * half;
        const int i0 = INTERLEAVED ? 2 * j : j;
        const int i1 = INTERLEAVED ? 2 * j + 1 : j + half;
        const double a = p * s_invf[j];
        const double nrev = rint(a * 0.15915494309189535);
        double red = fma(-nrev, 6.283185307179586, a);
        red = fma(-nrev, 2.4492935982947064e-16, red);
        float sn, cs;
        sincosf((float)red, &sn, &cs);
        const float x0 = __uint_as_float((uint32_t)qr[hq * D + i0] << 16);
        const float x1 = __uint_as_float((uint32_t)qr[hq * D + i1] << 16);
        s_q[hq * D + i0] = fmaf(x0, cs, -(x1 * sn));
        s_q[hq * D + i1] = fmaf(x1, cs, x0 * sn);
    }
    __syncthreads();

    const int G = Hq / H;
    const int upr = (H * D) >> 3;   // 16-byte units per K row
    const int lph = D >> 3;         // lanes (units) per head: a power of two <= 64
    const int64_t lstride = num_slots * upr;
    const int32_t* btr = block_table + (int64_t)r * max_blocks;
    float* out = scores + (int64_t)r * Hq * max_tokens;
    uint32_t flags = 0;
    for (int idx = blockIdx.x * kConsWaves + wave; idx < m; idx += gridDim.x * kConsWaves) {
        const int64_t pos = (int64_t)start_pos + idx;
        const int64_t blk = pos / page_size;
        if (blk >= max_blocks) { flags |= IS_DEV_BT_SHORT; continue; }
        const int32_t b = btr[blk];
        if (b < 0) { flags |= IS_DEV_BAD_BLOCK; continue; }
        const int64_t slot = (int64_t)b * page_size + pos % page_size;
        if (slot >= num_slots) { flags |= IS_DEV_SLOT_RANGE; continue; }
        const uint4* krow = paged_k + (int64_t)layer * lstride + slot * upr;
        for (int u0 = 0; u0 < upr; u0 += kWave) {
            const int u = u0 + lane;
            float part[kConsMaxG];
#pragma unroll
            for (int g = 0; g < kConsMaxG; ++g) part[g] = 0.f;
            int h = 0;
            if (u < upr) {
                const uint4 kv = krow[u];
                h = (u << 3) / D;
                const int e0 = (u << 3) - h * D;
                const uint32_t w[4] = {kv.x, kv.y, kv.z, kv.w};
                float k8[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    k8[2 * e] = bf16_lo(w[e]);
                    k8[2 * e + 1] = bf16_hi(w[e]);
                }
#pragma unroll
                for (int g = 0; g < kConsMaxG; ++g) {
                    if (g < G) {
                        const float* qg = s_q + (h * G + g) * D + e0;
                        float acc = 0.f;
#pragma unroll
                        for (int e = 0; e < 8; ++e) acc = fmaf(qg[e], k8[e], acc);
                        part[g] = acc;
                    }
                }
            }
            for (int off = 1; off < lph; off <<= 1)
#pragma unroll
                for (int g = 0; g < kConsMaxG; ++g) part[g] += __shfl_xor(part[g], off, kWave);
            if (u < upr && (lane & (lph - 1)) == 0) {
#pragma unroll
                for (int g = 0; g < kConsMaxG; ++g)
                    if (g < G) out[(int64_t)(h * G + g) * max_tokens + idx] = part[g];
            }
        }
    }
    if (flags) atomicOr(&s_flags, flags);
    __syncthreads();
    if (t == 0 && s_flags && status) atomicOr(status, s_flags);
}

int consumer_max_q_elems() { return kConsMaxQ; }
int consumer_max_group() { return kConsMaxG; }

hipError_t launch_paged_scores(const void* q, const int32_t* qpos, const void* paged_k,
                               int32_t layer, const int32_t* block_table, int32_t page_size,
                               int32_t start_pos, const int32_t* m, float* scores, int32_t nq,
                               int32_t Hq, int32_t H, int32_t D, int64_t num_slots,
                               int32_t max_blocks, int32_t max_tokens, float rope_theta,
                               const double* inv_freq, int32_t interleaved, uint32_t* status,
                               hipStream_t st) {
    if (max_tokens == 0) return hipSuccess;
    const int cus = compute_units();
    int64_t per_req = ((int64_t)max_tokens + kConsWaves - 1) / kConsWaves;
    const int64_t cap = (4LL * cus + nq - 1) / nq;
    if (per_req > cap) per_req = cap;
    if (per_req < 1) per_req = 1;
    dim3 grid((unsigned)per_req, (unsigned)nq);
    if (interleaved)
        hipLaunchKernelGGL(paged_scores_kernel<true>, grid, dim3(kConsThreads), 0, st,
                           (const uint16_t*)q, qpos, (const uint4*)paged_k, layer, block_table,
                           page_size, start_pos, m, scores, Hq, H, D, num_slots, max_blocks,
                           max_tokens, rope_theta, inv_freq, status);
    else
        hipLaunchKernelGGL(paged_scores_kernel<false>, grid, dim3(kConsThreads), 0, st,
                           (const uint16_t*)q, qpos, (const uint4*)paged_k, layer, block_table,
                           page_size, start_pos, m, scores, Hq, H, D, num_slots, max_blocks,
                           max_tokens, rope_theta, inv_freq, status);
    return hipGetLastError();
}

}  // namespace is
