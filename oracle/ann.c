/*
 * Plain CPU oracle for the graph-ANN retrieval backend: a proximity graph
 * over the fact embeddings and a beam search over it (§2.6, the GPU-resident
 * graph index the paper uses as its vector backend; §6.1: inner-product
 * similarity, 64 graph neighbours, beam width 64).
 *
 * TEST INFRASTRUCTURE ONLY, like oracle.c: loaded by the test suite, the
 * smoke check and the benchmark's CPU-baseline leg, never by the product
 * library, and sharing nothing with it.
 *
 * The paper names the index's parameters but not its construction or its
 * search loop; the readings taken here (listed with the design notes) are:
 *
 * Graph (out-degree R, h = floor(R/2)):
 *   F[i]   = the R facts j != i with the highest s(i, j) = <x_i, x_j>,
 *            best first, equal scores to the lower id (the exact R-nearest
 *            neighbour list under the retrieval order of §3.2);
 *   rev(i) = the facts j with i among F[j][0..h), ordered by the position
 *            of i in F[j], then by j;
 *   G[i]   = F[i][0..h), then the first facts of rev(i) not already listed,
 *            up to R - h of them, then F[i][h..R) in order, skipping facts
 *            already listed, until G[i] holds R facts.
 *   The reverse edges make every fact that some fact lists in its first h
 *   neighbours reachable from it (a forward-only nearest-neighbour graph
 *   leaves facts that nobody lists unreachable).
 *
 * Beam search (beam width B, search width P, at most T iterations):
 *   order: a fact ranks above another if its score is higher, or equal with
 *   a lower id (the same order as exact retrieval, §3.2);
 *   beam: the min(B, n_seeds) best seeds, none of them expanded;
 *   iteration: take the first P facts of the beam (in rank order) that are
 *   not expanded yet; if there are none, stop; mark them expanded; score
 *   every neighbour of theirs that is not in the beam (each once); the new
 *   beam is the B best of the old beam and these neighbours;
 *   result: the first k facts of the beam (id -1 and score -inf past its
 *   end); iterations = the number of iterations that expanded something.
 *
 * Scores are binary64 dot products of the decoded fp32/bf16 inputs.
 * Parity pins: the "not gpu" tests in test_oracle_ann.py (hand-worked
 * examples under tests/golden/, brute force, closed-form special cases).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ANN_F32 0
#define ANN_BF16 1
#define ANN_ID_RANGE 1u /* a graph entry or seed outside [0, n) */

static double ann_load(const void* base, int64_t idx, int32_t dtype)
{
    if (dtype == ANN_F32) return (double)((const float*)base)[idx];
    uint32_t bits = ((uint32_t)((const uint16_t*)base)[idx]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static double ann_dot(const void* a, int64_t ia, const void* b, int64_t ib, int32_t d,
                      int32_t dtype)
{
    double s = 0.0;
    for (int32_t t = 0; t < d; ++t) s += ann_load(a, ia + t, dtype) * ann_load(b, ib + t, dtype);
    return s;
}

typedef struct {
    double s;
    int64_t id;
    int expanded;
} ann_entry;

/* 1 if a ranks above b */
static int ann_above(double sa, int64_t ia, double sb, int64_t ib)
{
    return sa > sb || (sa == sb && ia < ib);
}

static int ann_cmp(const void* pa, const void* pb)
{
    const ann_entry* a = (const ann_entry*)pa;
    const ann_entry* b = (const ann_entry*)pb;
    if (ann_above(a->s, a->id, b->s, b->id)) return -1;
    if (ann_above(b->s, b->id, a->s, a->id)) return 1;
    return 0;
}

/* ---- forward lists: exact R nearest neighbours, self excluded ---------- */
int oracle_ann_knn(const void* bank, int64_t n, int32_t d, int32_t dtype, int32_t R, int32_t* F)
{
    if (!bank || !F || n < 2 || d < 1 || R < 1 || R > n - 1) return -1;
    if (dtype != ANN_F32 && dtype != ANN_BF16) return -1;
    ann_entry* all = (ann_entry*)malloc((size_t)n * sizeof(ann_entry));
    if (!all) return -2;
    for (int64_t i = 0; i < n; ++i) {
        int64_t c = 0;
        for (int64_t j = 0; j < n; ++j) {
            if (j == i) continue;
            all[c].s = ann_dot(bank, i * d, bank, j * d, d, dtype);
            all[c].id = j;
            all[c].expanded = 0;
            ++c;
        }
        qsort(all, (size_t)c, sizeof(ann_entry), ann_cmp);
        for (int32_t r = 0; r < R; ++r) F[i * R + r] = (int32_t)all[r].id;
    }
    free(all);
    return 0;
}

/* ---- final lists: forward half, reverse edges, forward fill ------------ */
typedef struct {
    int32_t pos;
    int32_t from;
} ann_rev;

static int ann_rev_cmp(const void* pa, const void* pb)
{
    const ann_rev* a = (const ann_rev*)pa;
    const ann_rev* b = (const ann_rev*)pb;
    if (a->pos != b->pos) return a->pos < b->pos ? -1 : 1;
    if (a->from != b->from) return a->from < b->from ? -1 : 1;
    return 0;
}

static int ann_listed(const int32_t* list, int32_t len, int32_t id)
{
    for (int32_t t = 0; t < len; ++t)
        if (list[t] == id) return 1;
    return 0;
}

int oracle_ann_merge(const int32_t* F, int64_t n, int32_t R, int32_t* G)
{
    if (!F || !G || n < 2 || R < 1 || R > n - 1) return -1;
    const int32_t h = R / 2;
    ann_rev* bucket = (ann_rev*)malloc((size_t)n * sizeof(ann_rev));
    if (!bucket) return -2;
    for (int64_t i = 0; i < n; ++i) {
        /* rev(i): every (position of i in F[j], j) with that position < h */
        int64_t nb = 0;
        for (int64_t j = 0; j < n; ++j)
            for (int32_t p = 0; p < h; ++p)
                if (F[j * R + p] == (int32_t)i) {
                    bucket[nb].pos = p;
                    bucket[nb].from = (int32_t)j;
                    ++nb;
                }
        qsort(bucket, (size_t)nb, sizeof(ann_rev), ann_rev_cmp);
        int32_t* out = G + i * R;
        int32_t len = 0;
        for (int32_t p = 0; p < h; ++p) out[len++] = F[i * R + p];
        for (int64_t b = 0; b < nb && len < R; ++b)
            if (!ann_listed(out, len, bucket[b].from)) out[len++] = bucket[b].from;
        for (int32_t p = h; p < R && len < R; ++p)
            if (!ann_listed(out, len, F[i * R + p])) out[len++] = F[i * R + p];
        if (len != R) { free(bucket); return -3; } /* cannot happen: F[i] is R distinct ids */
    }
    free(bucket);
    return 0;
}

int oracle_ann_build(const void* bank, int64_t n, int32_t d, int32_t dtype, int32_t R,
                     int32_t* F_out, int32_t* G)
{
    if (n < 2 || R < 1 || R > n - 1) return -1;
    int32_t* F = F_out ? F_out : (int32_t*)malloc((size_t)n * R * sizeof(int32_t));
    if (!F) return -2;
    int rc = oracle_ann_knn(bank, n, d, dtype, R, F);
    if (rc == 0) rc = oracle_ann_merge(F, n, R, G);
    if (!F_out) free(F);
    return rc;
}

/* ---- beam search -------------------------------------------------------- */
int oracle_ann_search(const void* query, int32_t nq, const void* bank, int64_t n, int32_t d,
                      int32_t dtype, const int32_t* graph, int32_t R, const int32_t* seeds,
                      int32_t n_seeds, int32_t B, int32_t P, int32_t k, int32_t max_iters,
                      int32_t* out_ids, double* out_scores, int32_t* out_iters, uint32_t* status)
{
    if (!query || !bank || !graph || !seeds || !out_ids || nq < 1 || n < 1 || d < 1) return -1;
    if (R < 1 || n_seeds < 1 || B < 1 || P < 1 || P > 64 || k < 1 || k > B || max_iters < 0)
        return -1;
    if (dtype != ANN_F32 && dtype != ANN_BF16) return -1;
    uint32_t flags = 0;
    const int64_t cap = (int64_t)B + (int64_t)P * R + n_seeds;
    ann_entry* pool = (ann_entry*)malloc((size_t)cap * sizeof(ann_entry));
    if (!pool) return -2;
    for (int32_t r = 0; r < nq; ++r) {
        const int64_t qoff = (int64_t)r * d;
        /* the beam starts as the best min(B, n_seeds) seeds */
        int64_t len = 0;
        for (int32_t s = 0; s < n_seeds; ++s) {
            const int64_t id = seeds[s];
            if (id < 0 || id >= n) { flags |= ANN_ID_RANGE; continue; }
            pool[len].s = ann_dot(query, qoff, bank, id * d, d, dtype);
            pool[len].id = id;
            pool[len].expanded = 0;
            ++len;
        }
        qsort(pool, (size_t)len, sizeof(ann_entry), ann_cmp);
        int64_t nb = len < B ? len : B;
        int32_t iters = 0;
        int64_t expand[64];
        while (iters < max_iters) {
            int32_t ne = 0;
            for (int64_t t = 0; t < nb && ne < P; ++t)
                if (!pool[t].expanded) {
                    pool[t].expanded = 1;
                    expand[ne++] = pool[t].id;
                }
            if (ne == 0) break;
            ++iters;
            /* neighbours not in the beam, each once, appended after it */
            int64_t total = nb;
            for (int32_t e = 0; e < ne; ++e)
                for (int32_t c = 0; c < R; ++c) {
                    const int64_t j = graph[expand[e] * R + c];
                    if (j < 0 || j >= n) { flags |= ANN_ID_RANGE; continue; }
                    int seen = 0;
                    for (int64_t t = 0; t < total && !seen; ++t) seen = pool[t].id == j;
                    if (seen) continue;
                    pool[total].s = ann_dot(query, qoff, bank, j * d, d, dtype);
                    pool[total].id = j;
                    pool[total].expanded = 0;
                    ++total;
                }
            qsort(pool, (size_t)total, sizeof(ann_entry), ann_cmp);
            nb = total < B ? total : B;
        }
        for (int32_t i = 0; i < k; ++i) {
            out_ids[(int64_t)r * k + i] = i < nb ? (int32_t)pool[i].id : -1;
            if (out_scores) out_scores[(int64_t)r * k + i] = i < nb ? pool[i].s : -INFINITY;
        }
        if (out_iters) out_iters[r] = iters;
    }
    free(pool);
    if (status) *status |= flags;
    return 0;
}
