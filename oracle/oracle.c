/*
 * Plain CPU oracle for the InferScale serving-time hot path:
 * exact top-k retrieval, reverse-proximity placement with prefix-sum slots,
 * and Chunked-RoPE injection of pre-RoPE keys and raw values into a paged
 * KV cache.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the reference that the GPU path is
 * checked against. Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load it. It shares no code, header, table or constant
 * with the HIP library, and the HIP library never calls it.
 *
 * Everything is computed the slow, obvious way, in binary64:
 *   - scores are plain dot products (§3.2, "Persistent memory store and
 *     retrieval": a top-k search by inner product over fact embeddings);
 *   - top-k is a full sort of every fact by (score desc, id asc);
 *   - placement follows §5.2 "Position policy": facts are laid out
 *     contiguously, the most relevant one last (adjacent to the query), and
 *     fact i starts at the cumulative length of the facts before it;
 *   - positions count from a caller-given start position (the instruction
 *     prefix of §3.3 occupies the positions before it);
 *   - slots follow the paged layout of §2.2 (fixed-size blocks from a pool,
 *     addressed through a per-request block table);
 *   - keys are rotated by the block-diagonal RoPE rotation R_p of §2.4 and
 *     Theorem "Chunked RoPE Injection" (§5.1), with frequencies
 *     theta^(-2j/D) for j < D/2, pairing element j with element j + D/2
 *     (the rotate-half convention of the Llama family, whose keys are taken
 *     before the model's own rotary step, §3.1); values are copied raw.
 *
 * bf16 values are handled as raw uint16 bit patterns. Decoding bf16 or fp32
 * to binary64 is exact; the only rounding to bf16 is the final
 * round-to-nearest-even of each rotated key element from binary64.
 *
 * Parity pins: every function here is pinned by the "not gpu" tests against
 * closed forms, brute force or an independent formulation (see the test
 * files named test_oracle_*.py).
 *
 * Threads: the scores, the top-k and the injection run their independent
 * outputs (one score, one query's ranking, one (token, layer) row) on an
 * OpenMP team of oracle_set_threads() threads (default: the OpenMP default,
 * i.e. OMP_NUM_THREADS or every core). Each output is still computed by one
 * thread in the order written below, so the results do not depend on the
 * thread count; one thread is the plain serial program.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1

/* data-dependent error flags, OR-ed into *status */
#define ORACLE_ID_RANGE 1u   /* an id < 0 or >= n                            */
#define ORACLE_BT_SHORT 2u   /* a position needs a block beyond max_blocks     */
#define ORACLE_CAPACITY 4u   /* placed tokens would exceed max_tokens          */
#define ORACLE_BAD_LEN 8u    /* a fact length < 0                              */
#define ORACLE_BAD_BLOCK 16u /* a block-table entry < 0                        */
#define ORACLE_SLOT_RANGE 32u /* a slot outside [0, num_slots)                 */
#define ORACLE_SRC_RANGE 64u /* a fact's rows fall outside [0, T_store)        */

/* ---- threads -------------------------------------------------------------- */

static int g_threads = 0; /* 0: the OpenMP default */

void oracle_set_threads(int32_t n) { g_threads = n > 0 ? n : 0; }

int32_t oracle_threads(void) { return g_threads > 0 ? g_threads : omp_get_max_threads(); }

/* ---- number formats ---------------------------------------------------- */

double oracle_bf16_to_double(uint16_t b)
{
    /* bf16 is the upper half of an IEEE binary32 pattern */
    uint32_t bits = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static double f32_to_double(float f) { return (double)f; }

/* Round a binary64 value to the nearest bf16, ties to even, directly (no
 * intermediate binary32 rounding). bf16 has 8 significant bits, exponents
 * down to -126 for normals and a fixed quantum of 2^-133 below that. */
uint16_t oracle_double_to_bf16(double x)
{
    if (isnan(x)) return (uint16_t)0x7FC0;
    uint16_t sign = signbit(x) ? (uint16_t)0x8000 : (uint16_t)0;
    double a = fabs(x);
    if (a == 0.0) return sign;
    if (isinf(a)) return (uint16_t)(sign | 0x7F80);
    int e;
    frexp(a, &e);            /* a = f * 2^e with f in [0.5, 1) */
    int E = e - 1;           /* a = 1.xxx * 2^E                */
    if (E < -126) E = -126;  /* subnormal range: fixed quantum */
    double quantum = ldexp(1.0, E - 7);
    double r = nearbyint(a / quantum) * quantum; /* a/quantum is exact */
    float rf = (float)r;     /* exact: r has at most 8 significant bits,
                                or overflows to +inf                */
    uint32_t bits;
    memcpy(&bits, &rf, sizeof bits);
    return (uint16_t)(sign | (uint16_t)(bits >> 16));
}

void oracle_double_to_bf16_n(const double* x, int64_t count, uint16_t* out)
{
    for (int64_t i = 0; i < count; ++i) out[i] = oracle_double_to_bf16(x[i]);
}

static double load_elem(const void* base, int64_t idx, int32_t dtype)
{
    if (dtype == ORACLE_F32) return f32_to_double(((const float*)base)[idx]);
    return oracle_bf16_to_double(((const uint16_t*)base)[idx]);
}

/* ---- step 1: similarity scores (§3.2) ------------------------------------
 * out[r][j] = sum_t query[r][t] * bank_r[j][t], in binary64.
 * bank_r = bank + r * bank_stride elements (bank_stride 0: one shared bank).
 * Every product of two decoded fp32 (or bf16) values is exact in binary64. */
int oracle_scores(const void* query, const void* bank, int64_t n, int32_t d,
                  int32_t nq, int64_t bank_stride, int32_t dtype, double* out)
{
    if (!query || !bank || !out || n < 0 || d < 1 || nq < 1) return -1;
    if (dtype != ORACLE_F32 && dtype != ORACLE_BF16) return -1;
    /* the queries decoded once (exact) */
    double* qd = (double*)malloc((size_t)nq * d * sizeof(double));
    if (!qd) return -2;
    for (int64_t i = 0; i < (int64_t)nq * d; ++i) qd[i] = load_elem(query, i, dtype);
    int failed = 0;
    /* one bank row per iteration, decoded (exactly) once for every query
     * that reads it; each score is summed over t = 0, 1, ... in order */
#pragma omp parallel num_threads(oracle_threads()) reduction(|:failed)
    {
        double* ed = (double*)malloc((size_t)d * sizeof(double));
        if (!ed) failed = 1;
#pragma omp for schedule(static)
        for (int64_t j = 0; j < n; ++j) {
            if (!ed) continue;
            for (int32_t r = 0; r < nq; ++r) {
                if (r == 0 || bank_stride != 0) {
                    const int64_t base = (int64_t)r * bank_stride + j * (int64_t)d;
                    for (int32_t t = 0; t < d; ++t) ed[t] = load_elem(bank, base + t, dtype);
                }
                const double* qr = qd + (int64_t)r * d;
                double s = 0.0;
                for (int32_t t = 0; t < d; ++t) s += qr[t] * ed[t];
                out[(int64_t)r * n + j] = s;
            }
        }
        free(ed);
    }
    free(qd);
    return failed ? -2 : 0;
}

/* ---- step 2: exact top-k by full sort (§3.2) -----------------------------
 * Rank order: higher score first; equal scores go to the lower id. */
typedef struct { double s; int64_t id; } scored_t;

static int by_score_desc_id_asc(const void* pa, const void* pb)
{
    const scored_t* a = (const scored_t*)pa;
    const scored_t* b = (const scored_t*)pb;
    if (a->s > b->s) return -1;
    if (a->s < b->s) return 1;
    if (a->id < b->id) return -1;
    if (a->id > b->id) return 1;
    return 0;
}

int oracle_topk(const double* scores, int64_t n, int32_t k, int32_t nq,
                int32_t* out_ids, double* out_scores)
{
    if (!scores || !out_ids || k < 1 || k > n || nq < 1) return -1;
    int failed = 0;
    /* one query's full sort per iteration */
#pragma omp parallel num_threads(oracle_threads()) reduction(|:failed)
    {
        scored_t* all = (scored_t*)malloc((size_t)n * sizeof(scored_t));
        if (!all) failed = 1;
#pragma omp for schedule(dynamic, 1)
        for (int32_t r = 0; r < nq; ++r) {
            if (!all) continue;
            for (int64_t j = 0; j < n; ++j) {
                all[j].s = scores[(int64_t)r * n + j];
                all[j].id = j;
            }
            qsort(all, (size_t)n, sizeof(scored_t), by_score_desc_id_asc);
            for (int32_t i = 0; i < k; ++i) {
                out_ids[(int64_t)r * k + i] = (int32_t)all[i].id;
                if (out_scores) out_scores[(int64_t)r * k + i] = all[i].s;
            }
        }
        free(all);
    }
    return failed ? -2 : 0;
}

/* ---- step 3: placement and slot map (§5.2 Position policy; §2.2) ----------
 * For request r with ranked ids[r][0..k-1] (best first):
 *   C_i = ids[k-1-i] when reverse_rank != 0 (most relevant next to the
 *         query), else C_i = ids[i];
 *   b_0 = 0, b_{i+1} = b_i + len(C_i), m = b_k;
 *   token t of C_i sits at position p = start_pos + b_i + t;
 *   slot(p) = block_table[r][p / page_size] * page_size + p % page_size.
 * Outputs per request r (rows of max_tokens): slots, positions, and
 * optionally the fact id and in-fact token index of each placed token.
 * A request with any data error gets m = 0, writes nothing else, and ORs a
 * flag into *status. */
int oracle_slot_map(const int32_t* ids, const int32_t* fact_lens, int32_t start_pos,
                    const int32_t* block_table, int32_t page_size,
                    int32_t k, int32_t nq, int64_t n, int64_t lens_stride,
                    int32_t max_blocks, int32_t max_tokens, int32_t reverse_rank,
                    int64_t* out_slots, int32_t* out_positions, int32_t* out_m,
                    int32_t* out_fact, int32_t* out_tok, uint32_t* status)
{
    if (!ids || !fact_lens || !block_table || !out_slots || !out_positions || !out_m)
        return -1;
    if (k < 1 || nq < 1 || page_size < 1 || start_pos < 0 || max_blocks < 0 || max_tokens < 0)
        return -1;
    uint32_t flags = 0;
    for (int32_t r = 0; r < nq; ++r) {
        const int32_t* rid = ids + (int64_t)r * k;
        const int32_t* lens = fact_lens + (int64_t)r * lens_stride;
        const int32_t* bt = block_table + (int64_t)r * max_blocks;
        uint32_t rflags = 0;
        int64_t total = 0;
        for (int32_t i = 0; i < k; ++i) {
            int32_t id = rid[i];
            if (id < 0 || id >= n) { rflags |= ORACLE_ID_RANGE; continue; }
            if (lens[id] < 0) { rflags |= ORACLE_BAD_LEN; continue; }
            total += lens[id];
        }
        if (!rflags && total > max_tokens) rflags |= ORACLE_CAPACITY;
        if (!rflags && total > 0) {
            int64_t last = (int64_t)start_pos + total - 1;
            if (last / page_size >= max_blocks) rflags |= ORACLE_BT_SHORT;
        }
        if (!rflags) {
            for (int64_t p = start_pos; p < start_pos + total; ++p)
                if (bt[p / page_size] < 0) { rflags |= ORACLE_BAD_BLOCK; break; }
        }
        if (rflags) {
            out_m[r] = 0;
            flags |= rflags;
            continue;
        }
        int64_t b = 0; /* b_i: tokens placed before fact C_i */
        for (int32_t i = 0; i < k; ++i) {
            int32_t c = reverse_rank ? rid[k - 1 - i] : rid[i];
            for (int32_t t = 0; t < lens[c]; ++t) {
                int64_t idx = b + t;
                int64_t p = (int64_t)start_pos + idx;
                int64_t slot = (int64_t)bt[p / page_size] * page_size + p % page_size;
                out_slots[(int64_t)r * max_tokens + idx] = slot;
                out_positions[(int64_t)r * max_tokens + idx] = (int32_t)p;
                if (out_fact) out_fact[(int64_t)r * max_tokens + idx] = c;
                if (out_tok) out_tok[(int64_t)r * max_tokens + idx] = t;
            }
            b += lens[c];
        }
        out_m[r] = (int32_t)total;
    }
    if (status) *status |= flags;
    return 0;
}

/* ---- step 4a: the RoPE rotation R_p of one head vector (§2.4, §5.1) -------
 * For j < D/2, with frequency w_j = theta^(-2j/D) and angle a = p * w_j:
 *   y[j]       = x[j] cos a - x[j + D/2] sin a
 *   y[j + D/2] = x[j + D/2] cos a + x[j] sin a
 * All in binary64. */
void oracle_rope_f64(const double* x, double p, double theta, int32_t D, double* y)
{
    int32_t half = D / 2;
    for (int32_t j = 0; j < half; ++j) {
        double w = pow(theta, -2.0 * (double)j / (double)D);
        double a = p * w;
        double c = cos(a), s = sin(a);
        double x0 = x[j], x1 = x[j + half];
        y[j] = x0 * c - x1 * s;
        y[j + half] = x1 * c + x0 * s;
    }
}

/* The same rotation with the model's own rotary table (§3.3: composition
 * applies RoPE with the model's rotary tables; §6.1: the evaluated models
 * differ in their RoPE parameterisation): pair j < D/2 is turned by the angle
 * a = p * inv_freq[j]. The pair is (j, j + D/2) in the half-split layout
 * (interleaved == 0) and (2j, 2j + 1) in the interleaved one. Binary64. */
void oracle_rope_table_f64(const double* x, double p, const double* inv_freq, int32_t D,
                           int32_t interleaved, double* y)
{
    int32_t half = D / 2;
    for (int32_t j = 0; j < half; ++j) {
        double a = p * inv_freq[j];
        double c = cos(a), s = sin(a);
        int32_t i0 = interleaved ? 2 * j : j;
        int32_t i1 = interleaved ? 2 * j + 1 : j + half;
        double x0 = x[i0], x1 = x[i1];
        y[i0] = x0 * c - x1 * s;
        y[i1] = x1 * c + x0 * s;
    }
}

/* The default table of the rotation above: inv_freq[j] = theta^(-2j/D). */
void oracle_default_inv_freq(double theta, int32_t D, double* inv_freq)
{
    for (int32_t j = 0; j < D / 2; ++j) inv_freq[j] = pow(theta, -2.0 * (double)j / (double)D);
}

void oracle_rope_table_bf16(const uint16_t* x, int64_t p, const double* inv_freq, int32_t D,
                            int32_t interleaved, uint16_t* y)
{
    double xd[1024], yd[1024];
    if (D < 2 || D > 1024 || D % 2) return;
    for (int32_t e = 0; e < D; ++e) xd[e] = oracle_bf16_to_double(x[e]);
    oracle_rope_table_f64(xd, (double)p, inv_freq, D, interleaved, yd);
    for (int32_t e = 0; e < D; ++e) y[e] = oracle_double_to_bf16(yd[e]);
}

/* bf16 head vector in, bf16 head vector out: decode, rotate in binary64,
 * round each element to nearest-even bf16. */
void oracle_rope_bf16(const uint16_t* x, int64_t p, double theta, int32_t D, uint16_t* y)
{
    double xd[1024], yd[1024];
    if (D < 2 || D > 1024 || D % 2) return;
    for (int32_t e = 0; e < D; ++e) xd[e] = oracle_bf16_to_double(x[e]);
    oracle_rope_f64(xd, (double)p, theta, D, yd);
    for (int32_t e = 0; e < D; ++e) y[e] = oracle_double_to_bf16(yd[e]);
}

/* ---- step 4b: composition + injection (§3.3, §3.4) ----------------------
 * For every request r, placed token idx < m[r] (fact C_i, in-fact token t,
 * re-derived from ids and fact_lens exactly as in oracle_slot_map), every
 * layer l and head h:
 *   src row  = fact_offsets[C_i] + t
 *   paged_k[l][slots[idx]][h][:] = R_{positions[idx]} preK[l][src][h][:]
 *   paged_v[l][slots[idx]][h][:] = V[l][src][h][:]      (bit copy)
 * Layouts: preK, V are [L][T_store][H][D]; pages are [L][num_slots][H][D];
 * all bf16. Nothing else in the pages is written. */
/* The same with the model's rotary table and pair layout: inv_freq [D/2]
 * (NULL: the default table of rope_theta) and interleaved as in
 * oracle_rope_table_f64. */
int oracle_inject_rotary(const int32_t* ids, const uint16_t* preK, const uint16_t* V,
                         const int64_t* slots, const int32_t* positions, double rope_theta,
                         uint16_t* paged_k, uint16_t* paged_v,
                         const int64_t* fact_offsets, const int32_t* fact_lens,
                         const int32_t* m, int32_t k, int32_t nq, int64_t n,
                         int64_t lens_stride, int32_t reverse_rank, int32_t max_tokens,
                         int32_t L, int32_t H, int32_t D, int64_t T_store, int64_t num_slots,
                         const double* inv_freq, int32_t interleaved, uint32_t* status)
{
    if (!ids || !preK || !V || !slots || !positions || !paged_k || !paged_v ||
        !fact_offsets || !fact_lens || !m)
        return -1;
    if (k < 1 || nq < 1 || L < 1 || H < 1 || D < 2 || D % 2 || D > 1024) return -1;
    double freq[512];
    if (inv_freq)
        for (int32_t j = 0; j < D / 2; ++j) freq[j] = inv_freq[j];
    else
        oracle_default_inv_freq(rope_theta, D, freq);
    uint32_t flags = 0;
    int64_t row = (int64_t)H * D;
    /* 1. the placement walk, in order: which stored row (or none) and which
     *    slot and position each placed token of each request takes */
    int64_t cap = 0;
    for (int32_t r = 0; r < nq; ++r) cap += m[r] < max_tokens ? (m[r] > 0 ? m[r] : 0) : max_tokens;
    int64_t* w_src = (int64_t*)malloc((size_t)(cap > 0 ? cap : 1) * sizeof(int64_t));
    int64_t* w_slot = (int64_t*)malloc((size_t)(cap > 0 ? cap : 1) * sizeof(int64_t));
    int64_t* w_pos = (int64_t*)malloc((size_t)(cap > 0 ? cap : 1) * sizeof(int64_t));
    if (!w_src || !w_slot || !w_pos) { free(w_src); free(w_slot); free(w_pos); return -2; }
    int64_t nw = 0;
    for (int32_t r = 0; r < nq; ++r) {
        const int32_t* rid = ids + (int64_t)r * k;
        const int32_t* lens = fact_lens + (int64_t)r * lens_stride;
        const int64_t* offs = fact_offsets + (int64_t)r * lens_stride;
        int32_t mr = m[r];
        if (mr > max_tokens) mr = max_tokens;
        int64_t b = 0;
        for (int32_t i = 0; i < k && b < mr; ++i) {
            int32_t c = reverse_rank ? rid[k - 1 - i] : rid[i];
            if (c < 0 || c >= n) { flags |= ORACLE_ID_RANGE; break; }
            int32_t len = lens[c];
            if (len < 0) { flags |= ORACLE_BAD_LEN; break; }
            int64_t off = offs[c];
            int src_ok = off >= 0 && off + len <= T_store;
            if (!src_ok) flags |= ORACLE_SRC_RANGE;
            for (int32_t t = 0; t < len && b + t < mr; ++t) {
                int64_t idx = b + t;
                int64_t slot = slots[(int64_t)r * max_tokens + idx];
                int64_t p = positions[(int64_t)r * max_tokens + idx];
                if (slot < 0 || slot >= num_slots) { flags |= ORACLE_SLOT_RANGE; continue; }
                if (!src_ok) continue;
                w_src[nw] = off + t;
                w_slot[nw] = slot;
                w_pos[nw] = p;
                ++nw;
            }
            b += len;
        }
    }
    /* 2. the writes: each (layer, head) takes every placed token in the
     *    walk's order, so a slot written twice ends as in a serial run */
#pragma omp parallel for collapse(2) schedule(dynamic, 1) num_threads(oracle_threads())
    for (int32_t l = 0; l < L; ++l) {
        for (int32_t h = 0; h < H; ++h) {
            for (int64_t e = 0; e < nw; ++e) {
                const int64_t so = ((int64_t)l * T_store + w_src[e]) * row + (int64_t)h * D;
                const int64_t dst = ((int64_t)l * num_slots + w_slot[e]) * row + (int64_t)h * D;
                oracle_rope_table_bf16(preK + so, w_pos[e], freq, D, interleaved, paged_k + dst);
                memcpy(paged_v + dst, V + so, (size_t)D * sizeof(uint16_t));
            }
        }
    }
    free(w_src);
    free(w_slot);
    free(w_pos);
    if (status) *status |= flags;
    return 0;
}

int oracle_inject(const int32_t* ids, const uint16_t* preK, const uint16_t* V,
                  const int64_t* slots, const int32_t* positions, double rope_theta,
                  uint16_t* paged_k, uint16_t* paged_v,
                  const int64_t* fact_offsets, const int32_t* fact_lens,
                  const int32_t* m, int32_t k, int32_t nq, int64_t n,
                  int64_t lens_stride, int32_t reverse_rank, int32_t max_tokens,
                  int32_t L, int32_t H, int32_t D, int64_t T_store, int64_t num_slots,
                  uint32_t* status)
{
    return oracle_inject_rotary(ids, preK, V, slots, positions, rope_theta, paged_k, paged_v,
                                fact_offsets, fact_lens, m, k, nq, n, lens_stride, reverse_rank,
                                max_tokens, L, H, D, T_store, num_slots, NULL, 0, status);
}

/* ---- the consumer of the pages: attention logits (Theorem "Chunked RoPE
 * Injection", §5.1; §3.4; §3.3: the query follows the memory) ----------------
 * For request r, query head hq (kv head hq / (Hq / H)), placed token idx <
 * m[r] at position p = start_pos + idx:
 *   scores[r][hq][idx] = sum_j (R_{qpos[r]} q[r][hq])_j * K[layer][slot(p)][hq/G][j]
 * with slot(p) = block_table[r][p / P] * P + p mod P, the rotation as in
 * oracle_rope_table_f64 (NULL table: rope_theta's default), in binary64 on
 * the decoded bf16 inputs. Tokens whose block is beyond max_blocks, negative,
 * or whose slot is outside the pool are skipped and flagged (BT_SHORT,
 * BAD_BLOCK, SLOT_RANGE); their scores are left untouched. */
int oracle_paged_scores(const uint16_t* q, const int32_t* qpos, const uint16_t* paged_k,
                        int32_t layer, const int32_t* block_table, int32_t page_size,
                        int32_t start_pos, const int32_t* m, double rope_theta,
                        const double* inv_freq, int32_t interleaved, int32_t nq, int32_t Hq,
                        int32_t H, int32_t D, int64_t num_slots, int32_t max_blocks,
                        int32_t max_tokens, double* scores, uint32_t* status)
{
    if (!q || !qpos || !paged_k || !block_table || !m || !scores) return -1;
    if (nq < 1 || H < 1 || Hq < H || Hq % H || D < 2 || D % 2 || D > 1024 || page_size < 1)
        return -1;
    double freq[512], xq[1024], rq[1024];
    if (inv_freq)
        for (int32_t j = 0; j < D / 2; ++j) freq[j] = inv_freq[j];
    else
        oracle_default_inv_freq(rope_theta, D, freq);
    const int32_t G = Hq / H;
    uint32_t flags = 0;
    for (int32_t r = 0; r < nq; ++r) {
        int32_t mr = m[r] < max_tokens ? m[r] : max_tokens;
        for (int32_t hq = 0; hq < Hq; ++hq) {
            const uint16_t* qv = q + ((int64_t)r * Hq + hq) * D;
            for (int32_t e = 0; e < D; ++e) xq[e] = oracle_bf16_to_double(qv[e]);
            oracle_rope_table_f64(xq, (double)qpos[r], freq, D, interleaved, rq);
            for (int32_t idx = 0; idx < mr; ++idx) {
                int64_t p = (int64_t)start_pos + idx;
                int64_t blk = p / page_size;
                if (blk >= max_blocks) { flags |= ORACLE_BT_SHORT; continue; }
                int32_t b = block_table[(int64_t)r * max_blocks + blk];
                if (b < 0) { flags |= ORACLE_BAD_BLOCK; continue; }
                int64_t slot = (int64_t)b * page_size + p % page_size;
                if (slot >= num_slots) { flags |= ORACLE_SLOT_RANGE; continue; }
                const uint16_t* kv =
                    paged_k + (((int64_t)layer * num_slots + slot) * H + hq / G) * D;
                double acc = 0.0;
                for (int32_t j = 0; j < D; ++j) acc += rq[j] * oracle_bf16_to_double(kv[j]);
                scores[((int64_t)r * Hq + hq) * max_tokens + idx] = acc;
            }
        }
    }
    if (status) *status |= flags;
    return 0;
}

