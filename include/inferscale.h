/*
 * inferscale.h -- C ABI of the MI355X (gfx950) retrieve + Chunked-RoPE
 * KV-inject library (libinferscale.so).
 *
 * The serving-time hot path of InferScale, as three calls:
 *   is_retrieve  exact top-k facts by inner product of a query embedding with
 *                a GPU-resident embedding bank (§3.2 "Persistent memory store
 *                and retrieval": the query embedding issues a top-k search
 *                that yields fact ids);
 *   is_slot_map  places the retrieved facts contiguously, most relevant fact
 *                adjacent to the query (§5.2 "Position policy"), and maps
 *                every placed token to its position and to its slot in a
 *                paged KV cache through the request's block table (§2.2
 *                paged blocks; §3.4 the scatter goes through the slot
 *                mapping);
 *   is_inject    gathers each placed token's stored pre-RoPE key and value,
 *                rotates the key to the token's position (§3.3 composition;
 *                §2.4 and Theorem "Chunked RoPE Injection", §5.1) and writes
 *                both into the paged cache (§3.4).
 * is_place_inject runs is_slot_map and is_inject as one launch, with the
 * same results.
 *
 * Conventions shared by every call
 *   - All data pointers are DEVICE pointers owned by the caller. The library
 *     allocates and frees nothing; retrieval scratch is the caller's
 *     workspace, sized by is_retrieve_workspace_size (is_retrieve_noalloc
 *     instead uses a fixed scratch array of the library's, for callers that
 *     cannot allocate).
 *   - `stream` is a hipStream_t (NULL: the legacy default stream). Every call
 *     only enqueues work on it and returns; none synchronizes. The calls keep
 *     no state between invocations and may run concurrently on different
 *     streams with disjoint outputs.
 *   - Return value: IS_OK, or a negative IS_ERR_* code for misuse detected on
 *     the host BEFORE anything is enqueued (null or misaligned pointers, bad
 *     sizes, unsupported dtype, short workspace), or IS_ERR_HIP when a launch
 *     fails. is_last_error() returns a message for the calling thread's last
 *     failure.
 *   - Errors that depend on device data (an id out of range, a block table
 *     that is too short, more tokens than max_tokens, ...) are reported by
 *     OR-ing IS_DEV_* flags into the caller's device word *status (which the
 *     caller clears). The offending request (slot map) or token/fact (inject)
 *     is skipped; nothing else about it is written.
 *   - bf16 is stored as raw 16-bit patterns (the upper half of an IEEE
 *     binary32).
 *   - Preconditions the library cannot check cheaply: the destination slots
 *     of one call are distinct (requests own disjoint blocks), and the page
 *     pools do not overlap the pre-RoPE store. Violations give unspecified
 *     page contents but no out-of-bounds access.
 */
#ifndef INFERSCALE_H
#define INFERSCALE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* return codes */
#define IS_OK 0
#define IS_ERR_INVALID (-1)      /* bad argument detected on the host        */
#define IS_ERR_UNSUPPORTED (-2)  /* valid but not supported by the library  */
#define IS_ERR_WORKSPACE (-3)    /* workspace missing or too small           */
#define IS_ERR_HIP (-4)          /* the HIP runtime refused a launch         */

/* element types of embeddings */
#define IS_DTYPE_F32 0
#define IS_DTYPE_BF16 1

/* device status flags, OR-ed into *status */
#define IS_DEV_ID_RANGE 1u    /* an id < 0 or >= n                                  */
#define IS_DEV_BT_SHORT 2u    /* a placed position needs a block index >= max_blocks */
#define IS_DEV_CAPACITY 4u    /* a request's facts hold more than max_tokens tokens  */
#define IS_DEV_BAD_LEN 8u     /* a fact length < 0                                  */
#define IS_DEV_BAD_BLOCK 16u  /* a block-table entry used by a request is < 0        */
#define IS_DEV_SLOT_RANGE 32u /* a slot outside [0, num_slots)                      */
#define IS_DEV_SRC_RANGE 64u  /* a fact's stored rows fall outside [0, T_store)      */

/* limits of the library */
#define IS_MAX_K 1024         /* largest k                                           */
#define IS_MAX_HEAD_DIM 512   /* largest head dimension D                            */

/* graph-ANN limits */
#define IS_ANN_MAX_DEGREE 128 /* out-degree of the proximity graph                   */
#define IS_ANN_MAX_BEAM 256   /* beam width                                          */
#define IS_ANN_MAX_WIDTH 4    /* beam entries expanded per iteration                 */
#define IS_ANN_MAX_EXPAND 256 /* width * degree                                      */

/* Library version string, e.g. "inferscale-gfx950 0.1.0". */
const char* is_version(void);

/* Message describing the calling thread's most recent IS_ERR_* return
 * ("" if none). The pointer stays valid until the thread's next call. */
const char* is_last_error(void);

/* Bytes of device workspace is_retrieve needs for these sizes (0 on bad
 * arguments; *bytes receives the size). Arguments as in is_retrieve. */
int is_retrieve_workspace_size(int64_t n, int32_t d, int32_t k, int32_t nq, int32_t dtype,
                               size_t* bytes);

/*
 * is_retrieve -- exact top-k by inner product (§3.2).
 *
 * For request r < nq with bank B_r = bank + r * bank_stride elements
 * (bank_stride == 0: every request searches the same bank):
 *   s_j = sum_t query_emb[r][t] * B_r[j][t],  j < n
 * accumulated in fp32 (bf16 inputs: exact bf16 x bf16 products, fp32 sums).
 * Output row r lists the k facts with the highest s_j, best first; equal
 * scores go to the lower id; -0.0 counts as +0.0 and NaN as the lowest.
 *
 *   query_emb  [nq][d] of dtype, 16-byte aligned
 *   bank       [n][d] (shared) or bank_stride-spaced [n][d] per request,
 *              row-major, 16-byte aligned, dtype as query_emb
 *   n          facts per bank, 1 <= n < 2^31
 *   d          embedding dimension, multiple of 8, 8 <= d <= 8192
 *   k          1 <= k <= min(n, IS_MAX_K)
 *   out_ids    [nq][k] int32 device
 *   out_scores [nq][k] fp32 device (may be NULL)
 *   nq         number of requests, >= 1
 *   bank_stride elements between consecutive requests' banks (0 = shared);
 *              a multiple of 8 elements
 *   dtype      IS_DTYPE_F32 or IS_DTYPE_BF16
 *   workspace  device scratch of at least is_retrieve_workspace_size bytes,
 *              256-byte aligned; its contents are not preserved
 */
int is_retrieve(const void* query_emb, const void* bank, int64_t n, int32_t d, int32_t k,
                int32_t* out_ids, float* out_scores, int32_t nq, int64_t bank_stride,
                int32_t dtype, void* workspace, size_t workspace_bytes, void* stream);

/* Largest scratch is_retrieve_noalloc uses (16 MiB per GPU). */
#define IS_RETRIEVE_NOALLOC_MAX_BYTES ((size_t)16 << 20)

/*
 * is_retrieve_noalloc -- is_retrieve for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): no workspace argument, and no allocation of any kind.
 *
 * Arguments, results and errors are those of is_retrieve (same kernels, same
 * output bits for the same inputs). Its scratch is a fixed array of
 * IS_RETRIEVE_NOALLOC_MAX_BYTES in the library's own device memory, one per
 * GPU, held from the first call on that GPU until the process ends; the
 * first call on a GPU looks up that array's device address (no allocation).
 * Sizes whose scratch (is_retrieve_workspace_size) exceeds the array are
 * refused with IS_ERR_WORKSPACE before anything is enqueued: for example
 * nq * n * 4 bytes of scores must fit (1 query: n up to ~4M; 8 queries over
 * 100,000 facts fit; the filtered matrix-core path for many queries over a
 * large bf16 bank does not).
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents: calls that overlap in time on one GPU (on different streams, or
 * from different threads) race and give undefined results. Calls on one
 * stream, one after another, are safe.
 */
int is_retrieve_noalloc(const void* query_emb, const void* bank, int64_t n, int32_t d, int32_t k,
                        int32_t* out_ids, float* out_scores, int32_t nq, int64_t bank_stride,
                        int32_t dtype, void* stream);

/*
 * is_slot_map -- placement and slot mapping (§5.2 Position policy; §2.2).
 *
 * For request r with ranked ids[r][0..k-1] (as is_retrieve returns them),
 * facts C_0..C_{k-1} are placed contiguously: C_i = ids[r][k-1-i] when
 * reverse_rank != 0 (the most relevant fact last, next to the query), else
 * C_i = ids[r][i]. With b_0 = 0 and b_{i+1} = b_i + len(C_i), token t of C_i
 * is placed token b_i + t at position p = start_pos + b_i + t, in slot
 *   block_table[r][p / page_size] * page_size + p % page_size.
 * Positions [0, start_pos) belong to the instruction prefix that precedes
 * the memory (§3.3) and are not touched.
 *
 *   ids            [nq][k] int32 device
 *   fact_lens      per-request [n] int32 tables, lens_stride elements apart
 *                  (lens_stride 0: one shared table)
 *   start_pos      first memory position, >= 0
 *   block_table    [nq][max_blocks] int32 device (physical block ids)
 *   page_size      tokens per block, >= 1
 *   out_slots      [nq][max_tokens] int64 device; entries >= m[r] untouched
 *   out_positions  [nq][max_tokens] int32 device; entries >= m[r] untouched
 *   out_m          [nq] int32 device: tokens placed (0 for a skipped request)
 *   k              1 <= k <= IS_MAX_K
 *   n              facts per table (ids must lie in [0, n))
 *   max_tokens     capacity per request row, >= 0
 *   reverse_rank   1: the paper's policy; 0: rank order as given
 *   status         device uint32 flag word (may be NULL)
 * A request with an id out of range, a negative length, more than
 * max_tokens tokens, or positions beyond its block table gets m = 0.
 */
int is_slot_map(const int32_t* ids, const int32_t* fact_lens, int32_t start_pos,
                const int32_t* block_table, int32_t page_size, int64_t* out_slots,
                int32_t* out_positions, int32_t* out_m, int32_t k, int32_t nq, int64_t n,
                int64_t lens_stride, int32_t max_blocks, int32_t max_tokens,
                int32_t reverse_rank, uint32_t* status, void* stream);

/*
 * is_inject -- fused gather + RoPE + scatter into the paged cache
 * (§3.3 composition; §3.4 injection; §2.4 / §5.1 rotation).
 *
 * For request r, placed token idx < m[r] (fact C_i, in-fact token t, derived
 * from ids, fact_lens and reverse_rank exactly as in is_slot_map), layer l,
 * head h:
 *   src = fact_offsets[r][C_i] + t
 *   paged_k[l][slots[r][idx]][h][:] = R_p preK[l][src][h][:], p = positions[r][idx]
 *   paged_v[l][slots[r][idx]][h][:] = V[l][src][h][:]           (bit copy)
 * R_p rotates pair (j, j + D/2) by the angle p * rope_theta^(-2j/D),
 * j < D/2. The angle is formed and reduced in fp64, its sine and cosine are
 * fp32, the rotation is fp32 and each output is rounded to nearest-even bf16.
 *
 *   preK, V        bf16 [L][T_store][H][D], 16-byte aligned: device memory of
 *                  the current device, or pinned host memory mapped into its
 *                  address space at the same address (hipHostMalloc), which
 *                  the kernel then reads over the host link -- the CPU-resident
 *                  KV store of §6.8 and App. C. Any other pointer is rejected
 *                  with IS_ERR_INVALID before anything is enqueued.
 *   slots, positions  [nq][max_tokens] as written by is_slot_map
 *   paged_k, paged_v  bf16 [L][num_slots][H][D] device, 16-byte aligned
 *   fact_offsets   per-request [n] int64 row offsets into the store
 *   fact_lens      per-request [n] int32 (both lens_stride elements apart)
 *   m              [nq] int32 device, tokens placed per request
 *   D              head dimension: a multiple of 16, <= IS_MAX_HEAD_DIM
 * Tokens whose slot lies outside [0, num_slots) and facts whose rows fall
 * outside the store are skipped and flagged.
 * Launch footprint: max(1, CUs / nq) workgroups of 768 threads per request,
 * each holding just over half of its CU's LDS (81 KiB of 160 KiB on MI355X)
 * so that it has its CU to itself; kernels on other streams can share those
 * CUs within the other half of the LDS and the remaining registers.
 */
int is_inject(const int32_t* ids, const void* preK, const void* V, const int64_t* slots,
              const int32_t* positions, float rope_theta, void* paged_k, void* paged_v,
              const int64_t* fact_offsets, const int32_t* fact_lens, const int32_t* m,
              int32_t k, int32_t nq, int64_t n, int64_t lens_stride, int32_t reverse_rank,
              int32_t max_tokens, int32_t L, int32_t H, int32_t D, int64_t T_store,
              int64_t num_slots, uint32_t* status, void* stream);

/* pair layouts of is_inject_rotary */
#define IS_ROPE_HALF_SPLIT 0  /* pairs (j, j + D/2): the rotate-half form (Llama, Mistral, Qwen) */
#define IS_ROPE_INTERLEAVED 1 /* pairs (2j, 2j + 1) */

/*
 * is_inject_rotary -- is_inject with the model's own rotary table and pair
 * layout (§3.3: composition applies RoPE with the model's rotary tables;
 * §6.1: the evaluated models differ in their RoPE parameterisation, e.g.
 * Llama 3.1's frequency scaling).
 *
 * Every argument of is_inject keeps its meaning, and:
 *   inv_freq  binary64 [D/2] device array, the angular frequency of pair j
 *             (radians per position): pair j of a token at position p turns
 *             by p * inv_freq[j]. NULL: rope_theta^(-2j/D), exactly as
 *             is_inject (rope_theta is then required to be positive and
 *             finite; with a table it is ignored). 8-byte aligned. Entries
 *             are not checked: a non-finite frequency gives non-finite keys.
 *   pairing   IS_ROPE_HALF_SPLIT or IS_ROPE_INTERLEAVED.
 * is_inject(...) is is_inject_rotary(..., NULL, IS_ROPE_HALF_SPLIT).
 */
int is_inject_rotary(const int32_t* ids, const void* preK, const void* V, const int64_t* slots,
                     const int32_t* positions, float rope_theta, void* paged_k, void* paged_v,
                     const int64_t* fact_offsets, const int32_t* fact_lens, const int32_t* m,
                     int32_t k, int32_t nq, int64_t n, int64_t lens_stride, int32_t reverse_rank,
                     int32_t max_tokens, int32_t L, int32_t H, int32_t D, int64_t T_store,
                     int64_t num_slots, const double* inv_freq, int32_t pairing, uint32_t* status,
                     void* stream);

/*
 * is_place_inject -- is_slot_map and is_inject_rotary as one launch (§5.2
 * placement and §2.2 slot mapping feeding the §3.4 injection; §3.3 and §5.1
 * rotation).
 *
 * For every request it computes exactly what is_slot_map followed by
 * is_inject_rotary computes: out_slots, out_positions and out_m as
 * is_slot_map writes them, and the same page contents and status flags.
 * The injection's set-up forms the placement offsets anyway, so each
 * token's slot is taken from the block table directly and the slot map's
 * separate launch (and its round trip through memory) is saved.
 *
 * Arguments: those of is_slot_map (start_pos, block_table, page_size,
 * max_blocks, out_slots, out_positions, out_m) and of is_inject_rotary
 * (the store, pages, rotary table and pair layout), with the same meaning,
 * layout, alignment and ownership; k, nq (<= 65535), n, lens_stride,
 * reverse_rank and max_tokens are shared. A request that is_slot_map would
 * skip (an id out of range, a negative length, more than max_tokens tokens,
 * positions beyond its block table, a negative block it uses) gets m = 0 and
 * no page is written for it; flags as for the two calls together.
 * Launch footprint: as is_inject's.
 */
int is_place_inject(const int32_t* ids, const void* preK, const void* V,
                    const int64_t* fact_offsets, const int32_t* fact_lens, int32_t start_pos,
                    const int32_t* block_table, int32_t page_size, int32_t max_blocks,
                    float rope_theta, const double* inv_freq, int32_t pairing, void* paged_k,
                    void* paged_v, int64_t* out_slots, int32_t* out_positions, int32_t* out_m,
                    int32_t k, int32_t nq, int64_t n, int64_t lens_stride, int32_t reverse_rank,
                    int32_t max_tokens, int32_t L, int32_t H, int32_t D, int64_t T_store,
                    int64_t num_slots, uint32_t* status, void* stream);

/*
 * is_paged_scores -- the consumer of the injected pages: attention logits of
 * each request's query against the keys of its placed tokens, read back
 * through the request's block table (Theorem "Chunked RoPE Injection", §5.1:
 * a key rotated at position p scores against a query at position N as the
 * stored key would at relative position p - N; §3.3: the query follows the
 * memory). For request r, query head hq, placed token idx < m[r]:
 *   pos   = start_pos + idx
 *   slot  = block_table[r][pos / page_size] * page_size + pos % page_size
 *   scores[r][hq][idx] = sum_j (R_qpos[r] q[r][hq])_j * paged_k[layer][slot][hq / (Hq/H)][j]
 * R rotates with inv_freq / pairing exactly as is_inject_rotary (NULL: the
 * default table of rope_theta); the query rotation uses fp64-reduced angles
 * and fp32 sine/cosine, the products and sums are fp32.
 *
 *   q            bf16 [nq][Hq][D] pre-RoPE queries, device
 *   qpos         int32 [nq] query positions (start_pos + m[r] for the
 *                position right after the memory)
 *   paged_k      bf16 [L][num_slots][H][D] as written by is_inject, 16-byte
 *                aligned; layer < L selects the layer
 *   block_table  int32 [nq][max_blocks]; m int32 [nq] (as for is_slot_map)
 *   scores       fp32 [nq][Hq][max_tokens], device; entries idx >= m[r] (and
 *                skipped tokens) are not written
 *   Hq           query heads: a multiple of H with Hq / H <= 8 and
 *                Hq * D <= 8192
 *   D            16, 32, 64, 128, 256 or 512
 * Tokens whose block lies beyond max_blocks, is negative or maps outside
 * [0, num_slots) are skipped and flagged (IS_DEV_BT_SHORT, IS_DEV_BAD_BLOCK,
 * IS_DEV_SLOT_RANGE).
 */
int is_paged_scores(const void* q, const int32_t* qpos, const void* paged_k, int32_t layer,
                    const int32_t* block_table, int32_t page_size, int32_t start_pos,
                    const int32_t* m, float* scores, int32_t nq, int32_t Hq, int32_t H, int32_t D,
                    int32_t L, int64_t num_slots, int32_t max_blocks, int32_t max_tokens,
                    float rope_theta, const double* inv_freq, int32_t pairing, uint32_t* status,
                    void* stream);

/*
 * is_stream_copy -- dst[0 .. bytes) = src[0 .. bytes), a streaming copy of
 * device memory (every byte read once and written once, non-temporal
 * 16-byte accesses, all CUs sweeping the buffers together). Not a step of
 * the method: the measured rate of this copy is the practical HBM ceiling
 * the inject's traffic (§3.5: every stored byte of the chosen facts read
 * once, every page byte written once) is reported against.
 *
 *   dst, src   device pointers, 16-byte aligned, not overlapping
 *   bytes      a multiple of 16 (0: nothing is enqueued)
 */
int is_stream_copy(void* dst, const void* src, size_t bytes, void* stream);

/*
 * Graph-ANN retrieval: the paper's vector backend is a GPU-resident
 * proximity graph over the fact embeddings, answered by a beam search on the
 * device (§2.6; §6.1: inner product, 64 neighbours, beam width 64). The
 * paper fixes those parameters only; the construction and the search loop
 * below are this library's reading. It is an alternative to is_retrieve for
 * banks too large to scan per request: the search reads the rows of the
 * facts it visits instead of the whole bank, and returns the exact top-k
 * only when the beam reaches it.
 *
 * Order: a fact ranks above another when its score (fp32 inner product, as
 * for is_retrieve) is higher, or equal with a lower id.
 */

/* Bytes of device workspace is_ann_build needs (0 on bad arguments). */
int is_ann_build_workspace_size(int64_t n, int32_t d, int32_t degree, int32_t dtype,
                                size_t* bytes);

/*
 * is_ann_build -- the proximity graph (out-degree R = degree, h = R / 2):
 *   F[i]   = the R facts j != i ranked highest for query x_i (exact, by the
 *            retrieval kernels of is_retrieve, k = R + 1 with i removed);
 *   rev(i) = the facts j with i among F[j][0 .. h), ordered by the position
 *            of i in F[j], then by j;
 *   G[i]   = F[i][0 .. h), then the first R - h facts of rev(i) that F[i]
 *            does not already list there, then F[i][h .. R) in order without
 *            the facts already listed, until R facts are listed.
 * The reverse edges keep facts that no forward list names reachable.
 * Seeds (entry points of the search): seed_ids[s] = floor(s * n / n_seeds)
 * and seed_bank[s] = bank[seed_ids[s]], a contiguous copy of their rows.
 *
 *   bank       [n][d] of dtype, 16-byte aligned; 2 <= n < 2^31;
 *              d a multiple of 8 in [8, 8192]
 *   degree     1 <= degree <= min(IS_ANN_MAX_DEGREE, n - 1)
 *   n_seeds    0 <= n_seeds <= n (0: seed_ids and seed_bank are not written
 *              and may be NULL)
 *   graph      int32 [n][degree] device (output G)
 *   fwd        int32 [n][degree] device (output F) or NULL
 *   seed_ids   int32 [n_seeds] device; seed_bank [n_seeds][d] of dtype,
 *              16-byte aligned
 *   workspace  at least is_ann_build_workspace_size bytes, 256-byte aligned
 * Cost: one exact retrieval per batch of 256 bank rows, then O(n * degree)
 * for the reverse edges. Built once per bank, outside the request path
 * (§6.1 counts index construction as offline set-up).
 */
int is_ann_build(const void* bank, int64_t n, int32_t d, int32_t degree, int32_t dtype,
                 int32_t n_seeds, int32_t* graph, int32_t* fwd, int32_t* seed_ids,
                 void* seed_bank, void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of device workspace is_ann_search needs (0 on bad arguments). */
int is_ann_search_workspace_size(int32_t n_seeds, int32_t d, int32_t beam, int32_t nq,
                                 int32_t dtype, size_t* bytes);

/*
 * is_ann_search -- beam search over the graph, per query r:
 *   the beam starts as the min(beam, n_seeds) best seeds (exact retrieval
 *   over seed_bank), none expanded; each iteration takes the first `width`
 *   unexpanded beam entries in rank order (none: stop), marks them
 *   expanded, scores every neighbour of theirs not in the beam (each once)
 *   and keeps the `beam` best of the old beam and those neighbours; at most
 *   max_iters iterations. Output row r: the first k beam entries, best
 *   first (id -1 and score -inf past the beam's end when it holds fewer
 *   than k), and out_iters[r] = iterations run.
 *
 *   query_emb  [nq][d] of dtype, 16-byte aligned; 1 <= nq <= 65535
 *   bank       [n][d] of dtype (the bank the graph was built on), 16-byte
 *              aligned; rows of at most 8 KiB (d <= 2048 fp32, 4096 bf16)
 *   graph      int32 [n][degree] (is_ann_build's G)
 *   seed_ids   int32 [n_seeds] distinct ids; seed_bank [n_seeds][d] their
 *              rows (is_ann_build's seeds); 1 <= n_seeds <= n
 *   beam       1 <= beam <= IS_ANN_MAX_BEAM; 1 <= k <= beam
 *   width      1 <= width <= IS_ANN_MAX_WIDTH, width * degree <=
 *              IS_ANN_MAX_EXPAND
 *   max_iters  >= 0 (0: the best seeds)
 * Scores: fp32 sums of the exact products; bf16 rows add two products per
 * packed dot step (round to nearest even, within about one ulp per step),
 * fp32 rows use fused multiply-adds.
 *   out_ids    int32 [nq][k]; out_scores fp32 [nq][k] or NULL; out_iters
 *              int32 [nq] or NULL; out_scored int32 [nq] or NULL: bank rows
 *              the search read for the query (each fact at most once while
 *              it is remembered as scored; the seed retrieval not counted);
 *              all device
 *   status     device flag word or NULL: a graph entry or seed id outside
 *              [0, n) sets IS_DEV_ID_RANGE and is skipped
 *   workspace  at least is_ann_search_workspace_size bytes, 256-byte aligned
 */
int is_ann_search(const void* query_emb, int32_t nq, const void* bank, int64_t n, int32_t d,
                  int32_t dtype, const int32_t* graph, int32_t degree, const int32_t* seed_ids,
                  const void* seed_bank, int32_t n_seeds, int32_t beam, int32_t width, int32_t k,
                  int32_t max_iters, int32_t* out_ids, float* out_scores, int32_t* out_iters,
                  int32_t* out_scored, uint32_t* status, void* workspace, size_t workspace_bytes,
                  void* stream);

#ifdef __cplusplus
}
#endif

#endif /* INFERSCALE_H */
