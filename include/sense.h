/*
 * sense.h -- C ABI of the SENSE retrieval + soft-gated evaluation hot path on
 * one AMD Instinct MI355X (gfx950).
 *
 * The method (SENSE: Semantic Embedding Navigation with Soft-gated
 * Evaluation) drafts tokens for speculative decoding by retrieving stored
 * continuations whose hidden-state keys are most similar to the target
 * model's current hidden state, then accepts a prefix of each draft with a
 * cascade of masks over the target model's logits.  This library implements
 * the data-parallel part of that loop:
 *
 *   sense_build_index       the datastore C_db of (key, continuation) pairs
 *                           (Sec. 3.1 Eq. 2; Sec. 3.2 Eq. 6)
 *   sense_retrieve          exact similarity scan + per-query top-k + gather
 *                           of each hit's continuation into a draft batch
 *                           (Sec. 3.1 Eq. 3; Sec. 3.2 Eqs. 7-8; Alg. 2's
 *                           L2Norm and retrieval steps)
 *   sense_soft_gate_verify  soft-gated evaluation of a draft batch against
 *                           aligned logits: accepted prefix length per draft
 *                           and the best draft per group
 *                           (Sec. 3.3 Eqs. 12-18; Alg. 4)
 *   sense_build_dynamic_index, sense_index_append
 *                           the dynamic context cache C_d and its update
 *                           (Sec. 3.2 Eq. 6; Alg. 1's retriever update;
 *                           Alg. 2's dynamic search is sense_retrieve on it)
 *   sense_select_candidates composite-score Top-N over the static and
 *                           dynamic hits with the anchor override
 *                           (Sec. 3.2 Eq. 8; Alg. 2)
 *   sense_build_loose_trie  LexSort and the loose trie of a draft pool: the
 *                           flattened tree, the map Gamma, the tree mask and
 *                           the static-KV mask (Sec. 3.2 Eq. 9; Alg. 2;
 *                           Alg. 3; App. tree attention mask)
 *   sense_soft_gate_verify_tree
 *                           soft-gated evaluation reading the flattened
 *                           tree's logits through Gamma (Sec. 3.2 Eq. 11;
 *                           Sec. 3.3; Alg. 4)
 *   sense_ivf_assign, sense_pq_encode, sense_build_ivf_index, sense_ivf_search
 *                           the inverted-file ANN retrieval the paper uses
 *                           (FAISS IVF-PQ of the implementation details):
 *                           IVF-Flat and IVF-PQ over the same top-k kernels
 *   sense_project           PCA projection + L2 normalisation of hidden
 *                           states: the query k = L2Norm(PCA(h)) of Alg. 2
 *                           and the projected datastore keys (Sec. 3.2
 *                           Eq. 6; App. implementation details)
 *
 * Conventions shared by every entry point
 *   - Pointers named keys, spans, span_len, queries, logits, drafts,
 *     draft_len, workspace and out_* are DEVICE pointers (HBM of the current
 *     HIP device).  Descriptor structs and size_t* results are host memory.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  All
 *     device work is enqueued on it and the call returns before it finishes:
 *     outputs are valid once the stream is synchronised, and inputs must stay
 *     alive and unchanged until then.
 *   - Arguments are validated on the host before anything is enqueued; a
 *     rejected call enqueues nothing and writes no output.  No C++ exception
 *     crosses this boundary.  sense_last_error_message() describes the last
 *     failure on the calling thread.
 *   - Conditions inside the data are defined results, not errors (a draft id
 *     outside [0, V), a zero-norm key, ties).
 *   - The library never synchronises the device except in
 *     sense_destroy_index (which frees device memory).
 */
#ifndef SENSE_H_
#define SENSE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The enumerations below are int-sized.  A C caller may pass any int where one
 * is expected (an unknown code is rejected with INVALID_ARGUMENT, or
 * described as "unknown" by sense_status_string); C++ sees each with int as
 * its fixed underlying type, so every int value is a valid value of it. */
#ifdef __cplusplus
#define SENSE_ENUM_BASE : int
#else
#define SENSE_ENUM_BASE
#endif

typedef enum SENSE_ENUM_BASE {
    SENSE_OK = 0,
    SENSE_ERR_INVALID_ARGUMENT = 1, /* NULL pointer, size out of range, mismatch */
    SENSE_ERR_MISALIGNED = 2,       /* pointer or stride breaks the 16-byte layout */
    SENSE_ERR_UNSUPPORTED = 3,      /* legal but outside what is implemented */
    SENSE_ERR_OUT_OF_MEMORY = 4,    /* a device allocation failed */
    SENSE_ERR_WORKSPACE = 5,        /* workspace NULL or smaller than required */
    SENSE_ERR_HIP = 6               /* the HIP runtime reported an error */
} sense_status_t;

typedef enum SENSE_ENUM_BASE { SENSE_F32 = 0, SENSE_F16 = 1, SENSE_BF16 = 2 } sense_dtype_t;

/* Similarity of Sec. 3.2 Eq. 8.  COSINE is the inner product of the
 * L2-normalised query and key (the paper L2-normalises both before search);
 * the key norms are those of the stored fp16/bf16 values. */
typedef enum SENSE_ENUM_BASE { SENSE_METRIC_IP = 0, SENSE_METRIC_COSINE = 1 } sense_metric_t;

/* Index flag: keep an owned, re-laid-out copy of the keys instead of
 * borrowing the caller's buffer (needed when the caller's row stride or base
 * address breaks the 16-byte layout). */
#define SENSE_INDEX_COPY_KEYS 1u

typedef struct sense_index sense_index_t; /* opaque host handle */

/* Datastore descriptor (Sec. 3.1 Eq. 2: pairs (k_i, c_i) with |c_i| <= M).
 *   keys       N x key_stride elements of key_dtype (F16 or BF16), row-major,
 *              row i's d elements contiguous.  Borrowed: must outlive the
 *              index unless SENSE_INDEX_COPY_KEYS.  Without the copy flag the
 *              base must be 16-byte aligned and key_stride % 8 == 0.
 *   n          number of rows, 1 <= n <= 2^31 - 1.
 *   d          key dimension, 1 <= d <= 8192 (the hidden sizes of the target
 *              models, or a projected dimension such as 64); d % 8 == 0.
 *              Keys of d <= 64 are scanned several rows per load
 *              instruction.
 *   key_stride elements between consecutive rows, >= d.
 *   spans      N x max_span int32 token ids: row i is the continuation c_i
 *              stored with key i.  Borrowed.
 *   max_span   M, 1 <= M <= 64.
 *   span_len   N int32 lengths in [0, M] (values outside are clamped), or
 *              NULL when every continuation is M tokens long.  Borrowed.
 *   metric     similarity used by sense_retrieve.
 *   flags      0 or SENSE_INDEX_COPY_KEYS. */
typedef struct {
    const void *keys;
    sense_dtype_t key_dtype;
    int64_t n;
    int32_t d;
    int64_t key_stride;
    const int32_t *spans;
    int32_t max_span;
    const int32_t *span_len;
    sense_metric_t metric;
    uint32_t flags;
} sense_index_desc_t;

/* Build an index over the datastore.  With one read of the keys, enqueued
 * on `stream`, it computes for COSINE the fp32 side table 1/||k_i|| (0 for a
 * zero row), for IP the largest fp32 ||k_i|| that is a number (it bounds the
 * error of the batched search's first pass, see sense_retrieve).  The index
 * owns only that table (N * 4 bytes) or value (4 bytes) and, with
 * SENSE_INDEX_COPY_KEYS, the key copy.  *out receives the handle; a static
 * index is immutable afterwards, so concurrent sense_retrieve calls on
 * different streams with separate workspaces are safe.
 * Errors: INVALID_ARGUMENT (NULL desc/out/keys/spans, sizes out of range,
 * non-key dtype), MISALIGNED, OUT_OF_MEMORY, HIP. */
sense_status_t sense_build_index(const sense_index_desc_t *desc, void *stream,
                                 sense_index_t **out);

/* Free the index and the device memory it owns (synchronises the device
 * first, so in-flight work that reads it completes).  NULL is a no-op. */
sense_status_t sense_destroy_index(sense_index_t *index);

/* Shape queries of an index (host values; any out pointer may be NULL).  For
 * a dynamic cache n is the number of rows appended so far. */
sense_status_t sense_index_info(const sense_index_t *index, int64_t *n, int32_t *d,
                                int32_t *max_span, sense_metric_t *metric,
                                sense_dtype_t *key_dtype);

/* Dynamic context cache (Sec. 3.2 Eq. 6: C_db = C_s u C_d; Alg. 1's
 * retriever update; Alg. 2's dynamic search).  For every generated position
 * p the cache holds the key that predicted token p and the token itself; the
 * continuation of row p is the generated text from p on, tokens[p .. p+M),
 * cut at the end of what has been appended (length min(M, n - p)).
 * sense_retrieve searches it exactly like a static index over its current n
 * rows.  The library owns all of its device memory:
 * capacity*d*2 bytes of keys, capacity*12 bytes of tokens, lengths and (for
 * COSINE) inverse norms.
 *   key_dtype  F16 or BF16 (appended keys are rounded to it, nearest-even).
 *   d          1 <= d <= 8192, d % 8 == 0.
 *   capacity   rows the cache can hold, 1 <= capacity <= 2^31 - 1.
 *   max_span   M, 1 <= M <= 64.
 *   metric     similarity used by sense_retrieve. */
typedef struct {
    sense_dtype_t key_dtype;
    int32_t d;
    int64_t capacity;
    int32_t max_span;
    sense_metric_t metric;
} sense_dynamic_index_desc_t;

/* Create an empty dynamic cache (n = 0); free it with sense_destroy_index.
 * Allocates synchronously and enqueues nothing.  Errors: INVALID_ARGUMENT,
 * OUT_OF_MEMORY. */
sense_status_t sense_build_dynamic_index(const sense_dynamic_index_desc_t *desc,
                                         sense_index_t **out);

/* Append `count` generated positions to a dynamic cache (Alg. 1's retriever
 * update R.Update(h, y)).
 *   keys       count x d elements of keys_dtype (F32, F16 or BF16),
 *              row-major and contiguous, element-aligned: row j is the
 *              hidden-state key that predicted tokens[j].
 *   tokens     count int32 token ids.
 *   count      >= 0 (0 is a no-op); n + count <= capacity.
 * The row count n grows when the call returns; the copy is enqueued on
 * `stream`.  A dynamic cache is the one mutable index: enqueue its appends
 * and the retrievals that read it on one stream (or order them with
 * events), because an append rewrites the continuation lengths of the last
 * M - 1 rows.  Errors: INVALID_ARGUMENT (not a dynamic cache, NULL pointers,
 * count < 0, capacity exceeded, unknown dtype), MISALIGNED, HIP. */
sense_status_t sense_index_append(sense_index_t *index, const void *keys,
                                  sense_dtype_t keys_dtype, const int32_t *tokens,
                                  int32_t count, void *stream);

/* Bytes of device workspace sense_retrieve needs for these sizes (for a
 * dynamic cache: at its capacity, so the size does not change as rows are
 * appended). */
sense_status_t sense_retrieve_workspace_size(const sense_index_t *index, int32_t n_queries,
                                             int32_t k, size_t *bytes);

/* Retrieval (Sec. 3.1 Eq. 3; Sec. 3.2 Eqs. 7-8; Alg. 2's L2Norm and search
 * steps), exact: for each query q,
 *   s[q, i] = sum_t q_t K[i, t]                    (IP)
 *   s[q, i] = that / (||q|| ||K_i||), 0 if a norm is 0   (COSINE)
 * accumulated in fp32 from the stored fp16/bf16 keys and the query as given;
 * the k rows with the largest s in the order (score desc, row index asc),
 * and their continuations.  One query is scored by fp32 FMA chains; a batch
 * of two or more on the matrix cores (an fp32 query as hi + lo halves of the
 * key type).  A batch of keys longer than 64 over more than 131072 rows
 * first takes every row's score from the query's hi half alone, keeps the
 * rows that a per-query bound on that score's error cannot exclude from the
 * top k, and returns fp32 rescores of those (the one-query arithmetic): the
 * same top k, with the one-query scan's rounding.
 *   queries      n_queries x d, dtype q_dtype (F32, or the key dtype),
 *                row-major, 16-byte aligned.
 *   n_queries    >= 1.   k: 1 <= k <= min(n, 1024) (an empty dynamic cache
 *                cannot be searched: skip it and pass n_dynamic = 0 to
 *                sense_select_candidates).
 *   out_ids      n_queries x k int64 row ids (required).
 *   out_scores   n_queries x k fp32 scores, or NULL.
 *   out_drafts   n_queries x k x max_span int32: spans[id][j] for
 *                j < span_len[id], -1 after; or NULL.
 *   out_draft_len n_queries x k int32 span lengths, or NULL.
 *   workspace    device scratch of at least sense_retrieve_workspace_size
 *                bytes, 256-byte aligned; its contents are not preserved.
 * Errors: INVALID_ARGUMENT, UNSUPPORTED (k > 1024; a batch of two or more
 * queries over a store so large that a query's candidate list, up to every
 * row plus 32 slots per scan wave, would pass 2^31 - 1 entries), MISALIGNED,
 * WORKSPACE, HIP.  An inverted-file index is searched with sense_ivf_search
 * instead (INVALID_ARGUMENT here). */
sense_status_t sense_retrieve(const sense_index_t *index, const void *queries,
                              sense_dtype_t q_dtype, int32_t n_queries, int32_t k,
                              int64_t *out_ids, float *out_scores, int32_t *out_drafts,
                              int32_t *out_draft_len, void *workspace,
                              size_t workspace_bytes, void *stream);

/* Retrieval for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation):
 * sense_retrieve with its scratch taken from a static device array inside the
 * library instead of a caller workspace.  Arguments, results and errors are
 * those of sense_retrieve, plus UNSUPPORTED when the call needs more than
 * sense_retrieve_noalloc_max_bytes() of scratch (64 MiB: e.g. one query over
 * up to ~15M rows, or 16 queries over 1M rows; use sense_retrieve with a
 * workspace beyond that).  It calls no allocator.  The device current on the
 * calling thread must be the one `stream` belongs to; each device has its own
 * copy of the array (held until the process ends), and its address is taken
 * once per device at the first call there.  Every call on a device shares
 * that device's array, which keeps the last call's contents: calls that may
 * overlap on one device (other streams, other threads) race and must be
 * serialised by the caller. */
sense_status_t sense_retrieve_noalloc(const sense_index_t *index, const void *queries,
                                      sense_dtype_t q_dtype, int32_t n_queries, int32_t k,
                                      int64_t *out_ids, float *out_scores, int32_t *out_drafts,
                                      int32_t *out_draft_len, void *stream);

/* Bytes of the static scratch sense_retrieve_noalloc draws on. */
size_t sense_retrieve_noalloc_max_bytes(void);

/* Soft-gate hyper-parameters (Alg. 4 inputs; Sec. 3.3; defaults of the
 * paper's experiments: gamma 0.05, top-k 3, W 6).
 *   gamma              entropy threshold: B_ent = I(E' > gamma)
 *   topk               k of the top-k membership mask, >= 1
 *   window             W of the look-ahead window, 0 <= W <= 64
 *   tau                window tolerance: B_con = I(R <= tau), tau >= 0
 *                      (0 is Alg. 4's R = 0)
 *   entropy_normalized 1: E' = E / ln|V| (Alg. 4); 0: E' = E in nats. */
typedef struct {
    float gamma;
    int32_t topk;
    int32_t window;
    int32_t tau;
    int32_t entropy_normalized;
} sense_gate_params_t;

/* Bytes of device workspace sense_soft_gate_verify needs for these sizes. */
sense_status_t sense_soft_gate_verify_workspace_size(int32_t n_cand, int32_t max_len,
                                                     int32_t vocab, size_t *bytes);

/* Soft-gated evaluation (Sec. 3.3 Eqs. 12-18; Alg. 4) of n_cand drafts.
 *   logits     n_cand x max_len rows of row_stride elements (F32, F16 or
 *              BF16); row (c, j) starts at element (c*max_len + j)*row_stride
 *              and is the target's distribution PREDICTING drafts[c][j] (the
 *              aligned rows of Sec. 3.2 Eq. 11: row 0 of every draft is the shared
 *              distribution at the current position).  Only rows with
 *              j < draft_len[c] are read.  Vector loads are used when the
 *              base is 16-byte aligned and row_stride*elem_size % 16 == 0.
 *   row_stride elements between rows, >= vocab.
 *   drafts     n_cand x max_len int32 token ids.
 *   draft_len  n_cand int32 in [0, max_len] (clamped), or NULL (= max_len).
 *   n_cand >= 0; 1 <= max_len <= 64; vocab >= 1; n_groups >= 1 divides
 *   n_cand: candidates [g*n_cand/n_groups, (g+1)*n_cand/n_groups) form group
 *   g (for instance the drafts retrieved for one query).
 * Per position (c, j < draft_len[c]), with x the row and t = drafts[c][j]:
 *   rank  = #{v : x_v > x_t} + #{v < t : x_v = x_t}  (V when t is outside
 *           [0, V)): t's place in the order (logit desc, index asc)
 *   B_em  = I(rank == 0)  (t is the first argmax of x)
 *   E     = -sum_v p_v ln p_v with p = softmax(x)
 *   B_ent = I(E' > gamma);  B_topk = I(rank < topk)
 * Per draft: B-bar = 1 - B_em, right-padded with W ones (positions
 * j >= draft_len count as mismatches); R[j] = sum_{u=1..W} B-bar[j+u];
 * B_con = I(R <= tau); G = B_em | (B_ent & (B_topk | B_con)), forced to 0 at
 * j >= draft_len; the accepted length n_c = number of leading ones of G.
 * Domain: logits are finite or -inf (a token of probability 0).  A +inf logit
 * still ranks exactly (the order above; equal +inf values by index), but
 * softmax of a row holding +inf is not a distribution of finite numbers: its
 * E' is NaN and B_ent 0.  NaN logits are outside the domain: such a row's
 * rank and gate bits are unspecified (every output stays in its range; the
 * call neither faults nor reads outside the row).
 * Outputs:
 *   out_accept_len n_cand int32, n_c in [0, draft_len[c]] (required).  The
 *                  paper's L of Alg. 4 is n_c - 1.
 *   out_best       n_groups int32: index within its group of the first draft
 *                  with the largest n_c (required).
 *   out_gate_score n_cand x max_len fp32 E' (0 at j >= draft_len), or NULL.
 *   out_masks      n_cand x max_len uint8 em | ent<<1 | topk<<2 | con<<3 |
 *                  G<<4 (em, ent, topk are 0 at j >= draft_len), or NULL.
 *   out_rank       n_cand x max_len int32 rank (V at j >= draft_len), or NULL.
 *   workspace      at least sense_soft_gate_verify_workspace_size bytes,
 *                  256-byte aligned; contents not preserved.
 * Errors: INVALID_ARGUMENT, MISALIGNED (workspace), WORKSPACE, HIP. */
sense_status_t sense_soft_gate_verify(const void *logits, sense_dtype_t logits_dtype,
                                      int64_t row_stride, const int32_t *drafts,
                                      const int32_t *draft_len, int32_t n_cand,
                                      int32_t max_len, int32_t vocab, int32_t n_groups,
                                      const sense_gate_params_t *params,
                                      int32_t *out_accept_len, int32_t *out_best,
                                      float *out_gate_score, uint8_t *out_masks,
                                      int32_t *out_rank, void *workspace,
                                      size_t workspace_bytes, void *stream);

/* Candidate-selection hyper-parameters (Sec. 3.2 Eq. 8; Alg. 2).  The
 * paper requires alpha >> beta and gives no values.
 *   alpha           weight of the first-token match I(D[i][0] == anchor)
 *   beta            weight of the similarity
 *   delta           boost added to every dynamic-cache similarity
 *   anchor_override 1: write the anchor into the first token of the first
 *                   and last selected drafts (Alg. 2); 0: leave them. */
typedef struct {
    float alpha;
    float beta;
    float delta;
    int32_t anchor_override;
} sense_select_params_t;

/* Candidate selection (Sec. 3.2 Eq. 8; Alg. 2's hybrid pool, composite
 * score, Top-N and anchor override) for n_queries queries at once.  Per query
 * q the pool D_all is its n_static static hits followed by its n_dynamic
 * dynamic-cache hits (the outputs of sense_retrieve on the two indexes), and
 * member i gets
 *   s_i = static score, or dynamic score + delta      (binary32 addition)
 *   S_i = fma(beta, s_i, I_i ? alpha : 0)              (binary32, one rounding)
 * with I_i = 1 when the draft's length is > 0 and its first token equals
 * anchors[q].  The top_n members by (S desc, position in D_all asc; NaN
 * scores last) are copied out; then, if anchor_override, the first token of
 * selected drafts 0 and top_n - 1 becomes anchors[q] (length at least 1).
 *   static_scores   n_queries x n_static fp32; static_drafts
 *                   n_queries x n_static x max_len int32; static_len
 *                   n_queries x n_static int32 or NULL (= max_len).
 *   dynamic_*       the same with n_dynamic (pointers may be NULL when
 *                   n_dynamic == 0).
 *   anchors         n_queries int32: the greedy token x~ of each query.
 *   n_static, n_dynamic >= 0 with 1 <= n_static + n_dynamic <= 2048;
 *   1 <= top_n <= n_static + n_dynamic; 1 <= max_len <= 64; n_queries >= 1.
 *   out_drafts      n_queries x top_n x max_len int32: the selected rows,
 *                   -1 past each length (required).
 *   out_len         n_queries x top_n int32 lengths clamped to [0, max_len]
 *                   (required).
 *   out_source      n_queries x top_n int32 position in D_all (< n_static:
 *                   static hit; else dynamic hit n_static + j), or NULL.
 *   out_score       n_queries x top_n fp32 composite scores S, or NULL.
 * Inputs are read, not modified.  Needs no workspace.  Errors:
 * INVALID_ARGUMENT (NULL required pointers, sizes out of range, NaN
 * parameters), UNSUPPORTED (pool above 2048), HIP. */
sense_status_t sense_select_candidates(const float *static_scores, const int32_t *static_drafts,
                                       const int32_t *static_len, int32_t n_static,
                                       const float *dynamic_scores,
                                       const int32_t *dynamic_drafts,
                                       const int32_t *dynamic_len, int32_t n_dynamic,
                                       const int32_t *anchors, int32_t n_queries,
                                       int32_t max_len, int32_t top_n,
                                       const sense_select_params_t *params,
                                       int32_t *out_drafts, int32_t *out_len,
                                       int32_t *out_source, float *out_score, void *stream);

/* Outputs of sense_build_loose_trie (all DEVICE pointers).  Per group g of
 * G = n_cand / n_groups drafts, the per-node arrays hold NODES = G * max_len
 * entries starting at g * NODES; tree nodes are numbered 0 .. L_g - 1 in
 * the order Alg. 3 extracts them (row-major over the sorted drafts, which
 * is a preorder of the tree); entries L_g .. NODES - 1 are set to -1.
 * Required:
 *   order       n_cand int32: order[g*G + r] = index within group g of its
 *               r-th draft in LexSort order.
 *   gamma       n_cand x max_len int32 in sorted order: the tree node of
 *               every position that exists (j < length), -1 elsewhere.
 *   tree_tokens, tree_parent, tree_depth, tree_cand
 *               n_groups x NODES int32: node u's token, its parent node (-1
 *               at depth 0), its depth (the draft position) and the first
 *               sorted draft whose path creates it (Gamma's inverse).
 *   tree_len    n_groups int32: L_g.
 * Optional (NULL = not written):
 *   sorted_drafts n_cand x max_len int32 (-1 past each length);
 *   sorted_len    n_cand int32 (clamped to [0, max_len]);
 *   mask          n_groups x NODES rows of mask_ld >= NODES uint8: row u,
 *                 columns v < L_g: 1 when v is on u's path (v = u
 *                 included), else 0; other entries untouched;
 *   full_mask     n_groups x NODES rows of cache_len elements of
 *                 full_mask_dtype (F32, F16 or BF16): row u < L_g is the
 *                 additive attention mask of tree token u over a static KV
 *                 cache whose first prefix_len positions hold the context
 *                 and the next L_g the tree: 0 where visible, -inf
 *                 elsewhere; rows >= L_g untouched. */
typedef struct {
    int32_t *order;
    int32_t *gamma;
    int32_t *tree_tokens;
    int32_t *tree_parent;
    int32_t *tree_depth;
    int32_t *tree_cand;
    int32_t *tree_len;
    int32_t *sorted_drafts;
    int32_t *sorted_len;
    uint8_t *mask;
    int64_t mask_ld;
    void *full_mask;
    sense_dtype_t full_mask_dtype;
    int32_t prefix_len;
    int64_t cache_len;
} sense_trie_t;

/* LexSort + loose trie of each group's drafts (Sec. 3.2 Eq. 9 and the tree
 * mask after it; Alg. 2's LexSort; Alg. 3; App. tree attention mask for a
 * static KV cache).
 *   drafts     n_cand x max_len int32 token ids (any values).
 *   draft_len  n_cand int32 lengths (clamped to [0, max_len]) or NULL
 *              (= max_len).  Positions j >= length do not exist: they match
 *              nothing and are no tree node.
 *   n_groups   >= 1, divides n_cand; G = n_cand / n_groups <= 1024 and
 *              G * max_len <= 4096; 1 <= max_len <= 64.
 * LexSort orders a group's drafts by their token sequences (signed int32
 * comparison; a proper prefix first; identical drafts by index).  Sorted
 * draft r's position j is shared when draft r-1 has the same tokens at
 * positions 0..j; every existing position that is not shared is a new tree
 * node.  The node count L_g is the number of distinct non-empty prefixes.
 * Errors: INVALID_ARGUMENT (NULL required pointers, sizes out of range,
 * mask_ld < NODES, unknown full_mask_dtype, prefix_len < 0, cache_len < 1),
 * UNSUPPORTED (group larger than 1024 drafts or 4096 tokens), HIP. */
sense_status_t sense_build_loose_trie(const int32_t *drafts, const int32_t *draft_len,
                                      int32_t n_cand, int32_t max_len, int32_t n_groups,
                                      const sense_trie_t *out, void *stream);

/* Bytes of device workspace sense_soft_gate_verify_tree needs. */
sense_status_t sense_soft_gate_verify_tree_workspace_size(int32_t n_cand, int32_t max_len,
                                                          int32_t vocab, int32_t n_groups,
                                                          size_t *bytes);

/* Soft-gated evaluation through the loose trie (Sec. 3.2 Eq. 11: the
 * aligned rows are [p_{t-1}; Gamma(P)]; Sec. 3.3 Eqs. 12-18; Alg. 4).
 *   logits     per group g, 1 + NODES rows of row_stride elements (F32, F16
 *              or BF16) starting at row g * (1 + NODES): row 0 is the
 *              distribution at the current position (p_{t-1}), row 1 + u the
 *              distribution after tree node u (P of the tree forward).  Only
 *              rows 0 and 1 + u for nodes with children are read.
 *   tree_tokens, tree_parent, tree_len, gamma
 *              as written by sense_build_loose_trie (n_groups x NODES,
 *              n_groups, n_cand x max_len).
 * Tree node u (u < L_g, parent in [-1, NODES)) is judged once, by row
 * 1 + parent(u) (row 0 at depth 0), with the statistics of
 * sense_soft_gate_verify; draft c's position j takes node gamma[c][j].  A
 * draft's length is its leading run of positions whose gamma is a judged
 * node; the gate, window, accepted length and best draft are then those of
 * sense_soft_gate_verify, per draft in gamma's (sorted) order: out_best is a
 * sorted position (order[] gives the original draft).  The outputs have the
 * layout of sense_soft_gate_verify's.  Needs n_cand % n_groups == 0 and the
 * group limits of sense_build_loose_trie.
 * Errors: INVALID_ARGUMENT, UNSUPPORTED, MISALIGNED (workspace), WORKSPACE,
 * HIP. */
sense_status_t sense_soft_gate_verify_tree(const void *logits, sense_dtype_t logits_dtype,
                                           int64_t row_stride, const int32_t *tree_tokens,
                                           const int32_t *tree_parent, const int32_t *tree_len,
                                           const int32_t *gamma, int32_t n_cand,
                                           int32_t max_len, int32_t vocab, int32_t n_groups,
                                           const sense_gate_params_t *params,
                                           int32_t *out_accept_len, int32_t *out_best,
                                           float *out_gate_score, uint8_t *out_masks,
                                           int32_t *out_rank, void *workspace,
                                           size_t workspace_bytes, void *stream);

/* A given PCA projection (the fit itself is not part of this library).
 *   mean       d_in fp32 (DEVICE), the mean subtracted first, or NULL.
 *   basis      d_out x d_in fp32 (DEVICE), row-major: row o is the o-th
 *              principal direction.
 *   d_in       1 <= d_in <= 8192, d_in % 8 == 0.
 *   d_out      1 <= d_out <= 256.
 *   normalize  1: L2-normalise every projected row (a zero row stays zero). */
typedef struct {
    const float *mean;
    const float *basis;
    int32_t d_in;
    int32_t d_out;
    int32_t normalize;
} sense_projection_t;

/* Bytes of device workspace sense_project needs (0 only for n_rows = 0). */
sense_status_t sense_project_workspace_size(const sense_projection_t *proj,
                                            sense_dtype_t x_dtype, int64_t n_rows,
                                            size_t *bytes);

/* Projection (Alg. 2: k = L2Norm(PCA(h)); Sec. 3.2 Eq. 6's Z applied to the
 * datastore keys; App. implementation details: 4096 -> 64 dims, then
 * L2-normalised):
 *   out[i][o] = sum_t (x[i][t] - mean[t]) * basis[o][t], accumulated in
 *   fp32, then out[i] /= ||out[i]|| if normalize, rounded to out_dtype
 *   (nearest-even).
 *   x          n_rows x d_in of x_dtype (F32, F16, BF16), row stride x_stride
 *              >= d_in elements, element-aligned.
 *   out        n_rows rows of out_stride >= d_out elements of out_dtype (F32,
 *              F16 or BF16); only the first d_out of each row are written.
 * 16-bit rows that are 16-byte aligned with x_stride % 8 == 0, 256 rows or
 * more, run as a matrix-core contraction (the basis split into a hi and a lo
 * half of the key type, ~16 mantissa bits for bf16, ~22 for fp16; up to 64
 * outputs the centring, normalisation and store happen in the same pass, so
 * the workspace holds no n_rows x d_out intermediate); other inputs run one
 * block per (row, output) in fp32.  Needs workspace (256-byte aligned,
 * sense_project_workspace_size bytes).
 * Errors: INVALID_ARGUMENT, MISALIGNED, WORKSPACE, HIP. */
sense_status_t sense_project(const sense_projection_t *proj, const void *x,
                             sense_dtype_t x_dtype, int64_t n_rows, int64_t x_stride, void *out,
                             sense_dtype_t out_dtype, int64_t out_stride, void *workspace,
                             size_t workspace_bytes, void *stream);

/* ---- Inverted file (the ANN retriever of Sec. 3.2 Eq. 7; App.
 * implementation details: FAISS IVF-PQ, nlist 4096, nprobe 32, pq_m 16).
 * The k-means fits of the coarse centroids and of the PQ codebooks are not
 * part of this library; assignment, encoding, the index layout and the search
 * are.  Key dimension d <= 128, d % 8 == 0 (the paper's keys are 64-dim). */

/* List of every key: the centroid it is most similar to under `metric`
 * (inner product, or cosine), accumulated in fp32; ties to the lower list.
 *   keys       n x d of key_dtype (F16/BF16), row stride key_stride.
 *   centroids  nlist x d fp32 (DEVICE), 1 <= nlist <= 65536.
 *   out_list   n int32 (DEVICE).
 * Errors: INVALID_ARGUMENT, MISALIGNED, HIP. */
sense_status_t sense_ivf_assign(const void *keys, sense_dtype_t key_dtype, int64_t n, int32_t d,
                                int64_t key_stride, const float *centroids, int32_t nlist,
                                sense_metric_t metric, int32_t *out_list, void *stream);

/* Product-quantisation codes of the residuals r_i = key_i - centroid[list_i]
 * (IVF-PQ): code j of key i = the entry of codebook j nearest to the j-th
 * d/m-dim slice of r_i (squared L2 in fp32, ties to the lower entry).
 *   codebooks  m x ksub x (d/m) fp32 (DEVICE); d % m == 0, d/m <= 16,
 *              1 <= ksub <= 256, ksub * d <= 16384.
 *   list_ids   n int32 (a list outside [0, nlist) gives code 0 throughout).
 *   out_codes  n x m uint8 (DEVICE).
 * Errors: INVALID_ARGUMENT, MISALIGNED, HIP. */
sense_status_t sense_pq_encode(const void *keys, sense_dtype_t key_dtype, int64_t n, int32_t d,
                               int64_t key_stride, const float *centroids, int32_t nlist,
                               const int32_t *list_ids, const float *codebooks, int32_t m,
                               int32_t ksub, uint8_t *out_codes, void *stream);

/* Inverted-file index descriptor.
 *   keys ... metric  as sense_index_desc_t; keys may be NULL for IVF-PQ.
 *   centroids        nlist x d fp32 (copied into the index).
 *   list_ids         n int32, every key's list (e.g. sense_ivf_assign).
 *   pq_codebooks     NULL: IVF-Flat (exact scores inside the probed lists);
 *                    else pq_m x pq_ksub x (d/pq_m) fp32 (copied), and
 *   pq_codes         n x pq_m uint8, every key's codes (e.g.
 *                    sense_pq_encode), values < pq_ksub. */
typedef struct {
    const void *keys;
    sense_dtype_t key_dtype;
    int64_t n;
    int32_t d;
    int64_t key_stride;
    const int32_t *spans;
    int32_t max_span;
    const int32_t *span_len;
    sense_metric_t metric;
    const float *centroids;
    int32_t nlist;
    const int32_t *list_ids;
    const float *pq_codebooks;
    int32_t pq_m;
    int32_t pq_ksub;
    const uint8_t *pq_codes;
} sense_ivf_desc_t;

/* Build an inverted-file index: each list's rows stored contiguously (the
 * keys for IVF-Flat, with their 1/||k|| for cosine; the codes for IVF-PQ)
 * with their original row ids.  The spans stay borrowed.  This call
 * synchronises `stream` once: it reads the list sizes back to size the
 * search buffers.  Errors: INVALID_ARGUMENT (also for list ids outside
 * [0, nlist) or codes >= pq_ksub, found on the device), MISALIGNED,
 * OUT_OF_MEMORY, HIP. */
sense_status_t sense_build_ivf_index(const sense_ivf_desc_t *desc, void *stream,
                                     sense_index_t **out);

/* Bytes of device workspace sense_ivf_search needs. */
sense_status_t sense_ivf_search_workspace_size(const sense_index_t *index, int32_t n_queries,
                                               int32_t k, int32_t nprobe, size_t *bytes);

/* Inverted-file search (Sec. 3.2 Eq. 7 with the paper's ANN retriever):
 *   coarse[l] = sim(q, centroid l) (IP, or cosine), in fp32;
 *   probes    = the nprobe lists with the largest coarse scores (ties: lower
 *               list id);
 *   each row of a probed list is scored: IVF-Flat as sense_retrieve scores
 *   it; IVF-PQ as u.c_l + sum_j LUT[j][code_j] with u = q (IP) or q/||q||
 *   (cosine), LUT[j][c] = u_j . codebook_j[c], summed in fp32 in the order
 *   j = 0..m-1, then added to u.c_l;
 *   the k best rows (score desc, original row asc), their continuations.
 * Fewer than k candidates: the tail has id -1, score NaN, an empty draft.
 *   queries    n_queries x d (F32 or the key dtype), 16-byte aligned.
 *   1 <= k <= 1024; 1 <= nprobe <= min(nlist, 1024).
 *   out_*      as sense_retrieve (out_ids required).
 *   out_probe  n_queries x nprobe int64 probed lists (best first), or NULL.
 * Errors: INVALID_ARGUMENT (also for an index that is not an inverted file),
 * UNSUPPORTED, MISALIGNED, WORKSPACE, HIP. */
sense_status_t sense_ivf_search(const sense_index_t *index, const void *queries,
                                sense_dtype_t q_dtype, int32_t n_queries, int32_t k,
                                int32_t nprobe, int64_t *out_ids, float *out_scores,
                                int32_t *out_drafts, int32_t *out_draft_len, int64_t *out_probe,
                                void *workspace, size_t workspace_bytes, void *stream);

/* Diagnostics for benchmarks and profilers.  Which part of the path a pair
 * of timing events brackets. */
typedef enum SENSE_ENUM_BASE {
    SENSE_TIMER_SCAN = 0,   /* similarity scan kernel(s) of sense_retrieve */
    SENSE_TIMER_TOPK = 1,   /* top-k selection + gather kernels of sense_retrieve */
    SENSE_TIMER_VERIFY = 2, /* both kernels of sense_soft_gate_verify(_tree) */
    SENSE_TIMER_SELECT = 3, /* the kernel of sense_select_candidates */
    SENSE_TIMER_TRIE = 4,   /* the kernels of sense_build_loose_trie */
    SENSE_TIMER_PROJECT = 5, /* the kernels of sense_project */
    SENSE_TIMER_IVF = 6,     /* the kernels of sense_ivf_search */
    SENSE_TIMER_FILTER = 7   /* the filtered full pass over the store of a
                                sampled-threshold batched sense_retrieve
                                (first group of 64 queries); a part of SCAN */
} sense_timer_t;

/* Register two hipEvent_t handles (created by the caller with timing
 * enabled) that the NEXT calls on this thread record, on their own stream,
 * immediately before and after the kernels named by `which`; NULL events
 * switch the timer off.  The setting is per calling thread and stays until
 * changed.  Events are only recorded, never waited on: read them with
 * hipEventElapsedTime after synchronising.  INVALID_ARGUMENT for an unknown
 * `which` or exactly one NULL event. */
sense_status_t sense_set_timer_events(sense_timer_t which, void *start_event, void *stop_event);

/* Diagnostic: one plain streaming read of `bytes` of device memory at `buf`
 * (16-byte non-temporal loads, a grid of 8 blocks of 256 threads per compute
 * unit, grid-stride, 8 loads in flight per thread), enqueued on `stream`.  It
 * measures the practical HBM read bandwidth of the device beside its
 * published peak; time it with events around the call.  `sink` is a device
 * word the kernel writes only in the (practically impossible) case that the
 * XOR of all words read equals a fixed constant, which keeps the loads alive.
 * buf 16-byte aligned, bytes a multiple of 16.  INVALID_ARGUMENT, MISALIGNED,
 * HIP. */
sense_status_t sense_read_bandwidth_probe(const void *buf, size_t bytes, uint32_t *sink,
                                          void *stream);

/* Static description of a status code. */
const char *sense_status_string(sense_status_t status);

/* Detail of the last failure on the calling thread ("" if none). */
const char *sense_last_error_message(void);

#ifdef __cplusplus
}
#endif

#endif /* SENSE_H_ */
