/*
 * pqhsa.h - C ABI of the PQ-HSA decode-attention operator for MI355X (gfx950).
 *
 * PQ-HSA ("hybrid sparse-approximate attention", arXiv 2609.33746) computes,
 * for each decode query, one approximate logit per indexed cached key from an
 * IVF-PQ index over key directions (Section 3.1, Eq. 2), attends the top-k of
 * those tokens plus a sink prefix and a local window exactly with their
 * original keys and values (Section 3.2, Eq. 3), and lets every unselected
 * indexed token enter the same softmax through its approximate logit, summed
 * per inverted list and multiplied by that list's value mean (Eq. 4). The
 * output is Eq. 5: y = (N_E + N_B) / (Z_E + Z_B).
 *
 * Conventions for every entry point
 *   - All functions return a pqhsa_status; no exception crosses the ABI.
 *     On failure pqhsa_last_error(ctx) holds a readable message.
 *   - Tensor arguments are device pointers owned by the caller unless stated
 *     otherwise; the caller keeps them alive until the work enqueued on
 *     `stream` has completed. Layouts are row-major, innermost index last.
 *   - B = batch, Hq / Hkv = query / KV heads, G = Hq / Hkv (the GQA group
 *     size; query head h reads KV head h / G, Section 3.3), d = head_dim,
 *     Nmax = max_seq, M = pq_m subspaces of d / M dimensions, K = pq_ksub
 *     codewords, n_list inverted lists.
 *   - Sequence b has N_b tokens. Its sink prefix is S = [0, n_sink), its local
 *     window L = [N_b - n_local, N_b) and its indexed region
 *     R_b = [n_sink, N_b - n_local) (Section 3.2). Index entries outside R_b
 *     are ignored. Between index updates the cache may grow past the index
 *     (pqhsa_set_lengths): L then spans every token after R_b.
 *   - One context serves one stream at a time: calls that overlap on
 *     different streams with the same context race on its workspace.
 */
#ifndef PQHSA_H
#define PQHSA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PQHSA_OK = 0,
    PQHSA_ERR_INVALID_ARGUMENT = 1, /* bad pointer, shape or value            */
    PQHSA_ERR_UNSUPPORTED = 2,      /* valid but not implemented (see shape)  */
    PQHSA_ERR_HIP = 3,              /* a HIP runtime call failed              */
    PQHSA_ERR_OUT_OF_MEMORY = 4,    /* device or host allocation failed       */
    PQHSA_ERR_NOT_PREPARED = 5      /* decode before pqhsa_index_prepare      */
} pqhsa_status;

typedef enum { PQHSA_F32 = 0, PQHSA_BF16 = 1 } pqhsa_dtype;

/* Problem shape, fixed for the life of a context.
 * Supported: head_dim = 128; (pq_m, pq_ksub) = (16, 256), 8-bit codes of
 * 8-dimensional subspaces, or (8, 16), the paper's own setting of 4-bit codes
 * of 16-dimensional subspaces (Section 3.1), kept as 4 bytes per token;
 * max_seq <= 2^20, 1 <= n_list <= 4096,
 * G in {1, 2, 4, 8}, 1 <= batch <= 256, kv_dtype F32 or BF16 (the query has
 * the same dtype as the cache), 0 <= max_topk <= max_seq, and
 * ceil((n_sink + n_local + 1024 + max_topk) / 128) + ceil(n_list / 64) <= 512
 * (1024: the growth of L between index updates). */
typedef struct {
    int32_t batch;
    int32_t n_q_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t max_seq;
    int32_t n_list;
    int32_t pq_m;
    int32_t pq_ksub;
    int32_t n_sink;   /* |S|, 4 in the paper's setting (Appendix A)   */
    int32_t n_local;  /* |L|, 128 in the paper's setting (Appendix A) */
    int32_t max_topk; /* largest k any decode call will ask for        */
    int32_t kv_dtype; /* pqhsa_dtype                                   */
} pqhsa_shape;

typedef struct pqhsa_ctx pqhsa_ctx;

/* Create a context: validates the shape and allocates, on the current HIP
 * device, the prepared-index storage and the whole decode workspace, so that
 * decode calls allocate nothing. *out receives the context (NULL on error).
 * Shape errors are reported before any HIP call is made. */
pqhsa_status pqhsa_create(const pqhsa_shape* shape, pqhsa_ctx** out);

/* Release every resource of the context (NULL is accepted). */
void pqhsa_destroy(pqhsa_ctx* ctx);

/* Load one prompt's IVF-PQ index into the context (Section 3.1, 3.3).
 *   seq_lens   HOST int32 [B]: N_b, with n_sink + n_local <= N_b <= max_seq.
 *   list_ids   int32 [B, Hkv, Nmax]          a_i, 0 <= a_i < n_list on R_b
 *   codes      uint8 [B, Hkv, Nmax, M]       z_im, one code per byte
 *                                             (< K; with K = 16 only the low
 *                                             four bits are kept)
 *   norms      float [B, Hkv, Nmax]          r_i (the key norm kept outside
 *                                             the quantizer)
 *   centroids  float [B, Hkv, n_list, d]     c_j
 *   codebooks  float [B, Hkv, M, K, d/M]     p_{m,z}
 *   list_means float [B, Hkv, n_list, d]     v_bar_j, the mean value over
 *                                             all of R_j (Eq. 4); 0 if empty
 * The context copies everything it needs and builds the list-major layout
 * on the device (a stable counting sort of R_b by list id), so the caller
 * may free these arrays once the call returns: the call synchronises
 * `stream` before returning. Returns INVALID_ARGUMENT, naming the first
 * offending (b, g, i), for a list id of R out of range (checked on the
 * device); the context is then left unprepared. */
pqhsa_status pqhsa_index_prepare(pqhsa_ctx* ctx, const int32_t* seq_lens,
                                 const int32_t* list_ids, const uint8_t* codes,
                                 const float* norms, const float* centroids,
                                 const float* codebooks, const float* list_means,
                                 hipStream_t stream);

/* Incremental index update (Section 3.3): the caches now hold
 * new_seq_lens[b] tokens (HOST int32 [B], each >= the current N_b and
 * <= max_seq, where N_b is the current length, see pqhsa_set_lengths). The
 * tokens that leave the local window, [n_sink + |R_b|, new N_b - n_local),
 * join R_b without re-clustering.
 *   - Each key k is stored as its norm r = ||k||, the list a of the centroid
 *     nearest to its direction u = k / r, and, per subspace, the index of
 *     the codeword nearest to that slice of u - c_a (Section 3.1). Distances
 *     are squared Euclidean in fp32; ties go to the smaller id; a zero key
 *     has r = 0.
 *   - The list means are refreshed over the grown lists (Eq. 4): the
 *     context keeps a float64 value sum per list, |R_j| v_bar_j from the
 *     last prepare or build plus every value added since, and each update
 *     writes sum / (n_old + n_new) in fp32 (the fp32 means never feed back,
 *     so many updates do not accumulate rounding).
 *   - The list-major layout becomes that of pqhsa_index_prepare over the
 *     grown lists (lists in increasing id, tokens in increasing id within a
 *     list), merged on the device: old members shift right, new ones append.
 * k_cache / v_cache / kv_strides as in pqhsa_decode (keys and values of
 * every token up to new_seq_lens). Equal lengths are a no-op rebuild.
 * Asynchronous: enqueues kernels on `stream`, allocates nothing. Host
 * checks first: INVALID_ARGUMENT for a length that shrinks or exceeds
 * max_seq. After a launch failure the index is unspecified until the next
 * successful prepare. */
pqhsa_status pqhsa_index_update(pqhsa_ctx* ctx, const int32_t* new_seq_lens,
                                const void* k_cache, const void* v_cache,
                                const int64_t* kv_strides, hipStream_t stream);

/* Build the index from the keys instead of taking one (Section 3.3 and the
 * appendix on the index build): k-means over every (sequence, KV head) at
 * once, then the context holds it as after pqhsa_index_prepare.
 *   - Each key of R_b is split into its norm (fp32) and direction u.
 *   - The coarse problem runs n_iter_coarse Lloyd iterations over the
 *     directions. Each iteration assigns every point to its nearest center
 *     (squared distance in fp32, ties to the smaller id), then moves each
 *     center to the float64 mean of its points. A center left without points
 *     takes the point farthest from its assigned center: the farthest first,
 *     ties to the smaller token id, one point per empty center in increasing
 *     center id.
 *   - Every token is then assigned to its list. Each of the M subspace
 *     problems runs n_iter_pq iterations over the residual slices
 *     (u - c_a)^(m), by the same rule.
 *   - Every token is then encoded against the trained model, and the list
 *     means are taken over the final lists.
 * The paper's setting is one coarse and two subspace iterations.
 *   seq_lens    HOST int32 [B]: N_b as in pqhsa_index_prepare
 *   k_cache, v_cache, kv_strides: as in pqhsa_decode
 *   init_coarse DEVICE int32 [B, Hkv, n_list]: token ids in R_b whose
 *               directions start the coarse centers (drawn by the caller)
 *   init_pq     DEVICE int32 [B, Hkv, M, K]: token ids in R_b whose residual
 *               slices start the codewords
 * Allocates and frees its own scratch (about 4 (M + 2) bytes per cache slot)
 * and synchronises `stream`. INVALID_ARGUMENT for a starting token outside
 * R_b or an iteration count outside [0, 64]. */
pqhsa_status pqhsa_index_build(pqhsa_ctx* ctx, const int32_t* seq_lens, const void* k_cache,
                               const void* v_cache, const int64_t* kv_strides,
                               const int32_t* init_coarse, const int32_t* init_pq,
                               int32_t n_iter_coarse, int32_t n_iter_pq, hipStream_t stream);

/* Set the current cache lengths N_b (HOST int32 [B]) between index updates
 * (Section 3.3: new tokens stay exact until the next update encodes them).
 * The tokens past R_b, [n_sink + |R_b|, N_b), form the exact tail L_b of
 * later decode calls, which grows from n_local to at most n_local + 1024.
 * Each N_b must lie in [indexed N_b, indexed N_b + 1024] and <= max_seq,
 * where the indexed N_b is the length of the last prepare or update (which
 * also reset the current lengths to it); otherwise INVALID_ARGUMENT. No
 * device work. */
pqhsa_status pqhsa_set_lengths(pqhsa_ctx* ctx, const int32_t* seq_lens);

/* Copy out the token-major index the context holds (synchronises `stream`);
 * any pointer may be NULL to skip that array. Entries of tokens outside R_b
 * are unspecified.
 *   list_ids   int32 [B, Hkv, max_seq]
 *   codes      uint8 [B, Hkv, max_seq, M], one code per byte
 *   norms      float [B, Hkv, max_seq]
 *   list_means float [B, Hkv, n_list, d]
 *   centroids  float [B, Hkv, n_list, d]
 *   codebooks  float [B, Hkv, M, K, d / M] */
pqhsa_status pqhsa_index_export_tokens(pqhsa_ctx* ctx, int32_t* list_ids, uint8_t* codes,
                                       float* norms, float* list_means, float* centroids,
                                       float* codebooks, hipStream_t stream);

/* One PQ-HSA decode step (Eqs. 2-5) for every (batch element, query head).
 *   q          [B, Hq, d] in kv_dtype, contiguous
 *   k_cache    keys   [B, Hkv, >= N_b, d] in kv_dtype
 *   v_cache    values, same layout and strides as k_cache
 *   kv_strides HOST int64 [3]: element strides of (b, kv head, token); the
 *              last dimension d must be contiguous
 *   topk       HOST int32 [B]: k_b = |T| for sequence b, 0 <= k_b <= |R_b|
 *              and k_b <= max_topk (k = ceil(rho |R|) in the paper)
 *   out        float [B, Hq, d]: y of Eq. 5, fp32
 * Asynchronous: enqueues kernels on `stream`, allocates nothing, never
 * synchronises. Requires a prior pqhsa_index_prepare. Device data are not
 * validated here. */
pqhsa_status pqhsa_decode(pqhsa_ctx* ctx, const void* q, const void* k_cache,
                          const void* v_cache, const int64_t* kv_strides,
                          const int32_t* topk, float* out, hipStream_t stream);

/* The same decode step with the budgets and lengths as DEVICE data, for a
 * caller that captures the step in a graph and replays it with new values
 * (Section 3.3: one step per generated token; the problem statement's
 * decode call takes N_b and k_b per step).
 *   q, k_cache, v_cache, kv_strides, out: as pqhsa_decode
 *   seq_lens   DEVICE int32 [B]: N_b of this step. The index covers R_b of
 *              the last prepare or update; tokens n_sink + |R_b| .. N_b - 1
 *              are the exact tail, at most n_local + 1024 of them.
 *   topk       DEVICE int32 [B]: k_b, 0 <= k_b <= min(|R_b|, max_topk)
 * Both arrays are read by the call's first kernel when the step runs, so a
 * captured graph takes the values present at each replay. Values outside
 * the ranges above are clamped on the device (not reported). The call
 * computes what pqhsa_decode computes for the same N_b and k_b (every
 * exact-set split of the partial buffer is launched; those past a row's
 * exact set exit at once). Asynchronous, allocates nothing, never
 * synchronises, records no stage timing. Requires a prior
 * pqhsa_index_prepare; INVALID_ARGUMENT for NULL arrays. */
pqhsa_status pqhsa_decode_device_args(pqhsa_ctx* ctx, const void* q, const void* k_cache,
                                      const void* v_cache, const int64_t* kv_strides,
                                      const int32_t* seq_lens, const int32_t* topk, float* out,
                                      hipStream_t stream);

/* pqhsa_decode reading a paged KV cache in place (the serving setting of
 * Section 4: vLLM-style pages named by a block table). Token t of sequence b
 * and KV head g sits at element
 *   block_table[b * max_blocks + t / page_size] * page_strides[0]
 *   + g * page_strides[1] + (t % page_size) * page_strides[2]
 * of k_pages (keys) and of v_pages (values); the last dimension d is
 * contiguous. An interleaved page layout [pages, Hkv, page_size, 2d] is
 * passed as k_pages = base, v_pages = base + d with page_strides
 * (Hkv * page_size * 2d, page_size * 2d, 2d).
 *   block_table DEVICE int32 [B, max_blocks]: page index of each logical
 *               block; entries past a sequence's last block are not read.
 *               The page indices are not validated.
 *   page_size   a power of two in [1, 2^20]; max_blocks * page_size must
 *               cover the longest prepared sequence.
 * Other arguments, and the result, as in pqhsa_decode (bit-identical to it
 * on the same rows). Asynchronous; allocates nothing. */
pqhsa_status pqhsa_decode_paged(pqhsa_ctx* ctx, const void* q, const void* k_pages,
                                const void* v_pages, const int64_t* page_strides,
                                const int32_t* block_table, int32_t max_blocks,
                                int32_t page_size, const int32_t* topk, float* out,
                                hipStream_t stream);

/* pqhsa_decode plus diagnostics for parity checks (synchronises `stream`).
 *   selected            int32 [B, Hq, max_topk] or NULL: the token ids of T,
 *                       ascending, padded with -1
 *   unselected_per_list int32 [B, Hq, n_list] or NULL: |B n R_j| (Eq. 4)
 *   scores              float [B, Hq, Nmax] or NULL: the approximate logit of
 *                       Eq. 2 for every token of R_b by token id, NaN
 *                       elsewhere (computed by the same device code as the
 *                       scan)
 * Returns PQHSA_ERR_UNSUPPORTED when selected or unselected_per_list is
 * requested and some k_b exceeds 8192. */
pqhsa_status pqhsa_decode_debug(pqhsa_ctx* ctx, const void* q, const void* k_cache,
                                const void* v_cache, const int64_t* kv_strides,
                                const int32_t* topk, float* out, int32_t* selected,
                                int32_t* unselected_per_list, float* scores,
                                hipStream_t stream);

/* Dense decode attention over the whole cache, y = sum_i e_i v_i / sum_i e_i
 * with e_i = exp(q.k_i / sqrt(d)) (Section 3, first paragraph): the same-chip
 * baseline. Arguments as in pqhsa_decode; seq_lens is a HOST int32 [B] with
 * 1 <= N_b <= max_seq. Needs no prepared index. Asynchronous. */
pqhsa_status pqhsa_dense_decode(pqhsa_ctx* ctx, const void* q, const void* k_cache,
                                const void* v_cache, const int64_t* kv_strides,
                                const int32_t* seq_lens, float* out,
                                hipStream_t stream);

/* Dense decode attention as pqhsa_dense_decode, without a context and
 * without allocating device memory: for callers that cannot allocate (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).
 *   batch, n_q_heads, n_kv_heads  the shape (G = n_q_heads / n_kv_heads in
 *                                 {1, 2, 4, 8}, batch <= 256)
 *   head_dim                      128
 *   kv_dtype                      PQHSA_F32 or PQHSA_BF16 (q, k_cache, v_cache)
 *   q, k_cache, v_cache, kv_strides, out  as in pqhsa_dense_decode
 *   seq_lens                      HOST int32 [batch], 1 <= N_b <= 2^20
 * Scratch: the split partials of every row, batch * n_q_heads *
 * ceil(max N_b / 2048) of 528 bytes each, live in one fixed 32 MiB device
 * array of the library (a copy on every GPU it runs on, held until the
 * process ends; its address is looked up on the first call on each device).
 * A call that needs more (for example batch * n_q_heads > 992 at
 * N_b = 131072) returns PQHSA_ERR_INVALID_ARGUMENT before any device work.
 * Nothing in the array needs to start at zero: every partial a call reads it
 * writes first. Every call on one GPU shares that GPU's array, so calls that
 * overlap on one GPU (other streams, other threads) race on it.
 * Asynchronous; enqueues two kernels on `stream`. Errors are reported by
 * pqhsa_last_error(NULL) on the calling thread. */
pqhsa_status pqhsa_dense_decode_noalloc(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                        int32_t head_dim, int32_t kv_dtype, const void* q,
                                        const void* k_cache, const void* v_cache,
                                        const int64_t* kv_strides, const int32_t* seq_lens,
                                        float* out, hipStream_t stream);

/* Copy out the prepared list-major layout (synchronises `stream`):
 *   perm    int32 [B, Hkv, Nmax]: token id at each list-major position of R_b
 *           (lists in increasing id, tokens in increasing id within a list),
 *           -1 past |R_b|
 *   offsets int32 [B, Hkv, n_list + 1]: start of each list in that order */
pqhsa_status pqhsa_index_export(pqhsa_ctx* ctx, int32_t* perm, int32_t* offsets,
                                hipStream_t stream);

/* Options (values are int64):
 *   PQHSA_OPT_FORCE_FALLBACK  1: every row takes the exact re-scan path of the
 *                             top-k stage (normally used only when the
 *                             sampled threshold yields fewer than k
 *                             candidates); for testing that path.
 *   PQHSA_OPT_STAGE_TIMING    1: record HIP events around the kernel of each
 *                             stage of each decode call (read with
 *                             pqhsa_stage_times).
 *   PQHSA_OPT_THRESHOLD_BIAS  added (as value / 1000.0) to every sampled
 *                             candidate threshold; a large value starves the
 *                             candidate set and forces the fallback.
 *   PQHSA_OPT_VARIANT         the background term (the mechanism variants of
 *                             Appendix B, on the same exact set):
 *                             PQHSA_VARIANT_B (default) per-list value means,
 *                             Eq. 4; PQHSA_VARIANT_T no background (softmax
 *                             over E alone); PQHSA_VARIANT_C every list takes
 *                             the global value mean over R_b (computed at
 *                             prepare as sum_j |R_j| v_bar_j / |R_b|, which is
 *                             the mean of the values over R_b when the list
 *                             means are the means over R_j);
 *                             PQHSA_VARIANT_BX list j takes the mean of its
 *                             unselected members, (|R_j| v_bar_j - sum of v_i
 *                             over T n R_j) / |B n R_j|, its weights formed
 *                             by the top-k stage. Under
 *                             PQHSA_VARIANT_T a row whose exact set is empty
 *                             (no sink, no window, k = 0) has no defined
 *                             output: its entries are NaN (0 / 0). Any other
 *                             value is PQHSA_ERR_INVALID_ARGUMENT. */
enum {
    PQHSA_OPT_FORCE_FALLBACK = 1,
    PQHSA_OPT_STAGE_TIMING = 2,
    PQHSA_OPT_THRESHOLD_BIAS = 3,
    PQHSA_OPT_VARIANT = 4
};
enum { PQHSA_VARIANT_B = 0, PQHSA_VARIANT_T = 1, PQHSA_VARIANT_C = 2, PQHSA_VARIANT_BX = 3 };
pqhsa_status pqhsa_set_option(pqhsa_ctx* ctx, int32_t option, int64_t value);

/* Stage durations (ms) of the last decode call made with stage timing on, in
 * launch order: [0] LUT build + threshold sample, [1] code scan,
 * [2] top-k select, [3] exact attention + background, [4] merge. Each is the
 * execution time of that stage's kernel (events recorded by the kernel
 * launch itself), without the gaps between launches.
 * `n` is the capacity of `ms`; *n_out receives the number of stages.
 * Synchronises on the recorded events. */
pqhsa_status pqhsa_stage_times(pqhsa_ctx* ctx, float* ms, int32_t n, int32_t* n_out);

/* Static description of a status code. */
const char* pqhsa_status_string(pqhsa_status status);

/* Message of the last failed call on this context ("" if none; NULL ctx gives
 * the message of the last failed call made without a context on this thread:
 * pqhsa_create or pqhsa_dense_decode_noalloc). */
const char* pqhsa_last_error(const pqhsa_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* PQHSA_H */
