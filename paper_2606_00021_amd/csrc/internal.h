// Internal declarations shared by the host layer and the kernel files of the
// SENSE hot-path library.  Nothing here is part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sense {

// Element encodings (same numbering as sense_dtype_t).
enum : int { DT_F32 = 0, DT_F16 = 1, DT_BF16 = 2 };

// Rows of the similarity scan handled by one 16-byte load of one lane:
// eight 2-byte key elements.  A wave (64 lanes) covers 512 elements of a row
// per load instruction.
constexpr int kLaneElems = 8;
constexpr int kWaveElems = 64 * kLaneElems;
constexpr int kMaxDim = 8192;       // 16 chunks of 512 elements per lane
// Verification launches one 256-thread block per judged row along the grid's
// x dimension, and one dispatch holds fewer than 2^32 work-items per
// dimension: at most this many (candidate, position) rows per call.
constexpr int kVerifyRowThreads = 256;
constexpr int64_t kMaxVerifyRows = (((int64_t)1 << 32) / kVerifyRowThreads) - 1;
constexpr int kMaxK = 1024;         // largest retrieval top-k
constexpr int kMaxLen = 64;         // longest draft
constexpr int kSelectChunk = 8192;  // elements per top-k selection block
constexpr int kMaxPool = 2048;      // largest static + dynamic candidate pool
constexpr int kMaxGroup = 1024;     // largest candidate group of the loose trie
constexpr int kMaxNodes = 4096;     // largest group x draft length of the loose trie
constexpr int kMaxProjOut = 256;    // largest projected dimension
constexpr int kProjMfmaMinRows = 256;   // 16-bit projections of this many rows use MFMA
constexpr int kSmallDim = 64;       // keys this short use the short-row scan
constexpr int kMaxIvfDim = 128;     // largest key dimension of an inverted-file index
constexpr int kMaxDsub = 16;        // largest PQ sub-vector
constexpr int kMaxNlist = 65536;    // most inverted lists

// Order-preserving map of an fp32 score to an unsigned key: larger score ->
// larger key; every NaN -> 0 (below everything); -0 is folded onto +0.
__host__ __device__ inline uint32_t score_key(float s) {
    if (s != s) return 0u;
    s = s + 0.0f;
    uint32_t u;
    __builtin_memcpy(&u, &s, 4);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__host__ __device__ inline float key_score(uint32_t k) {
    uint32_t u = (k & 0x80000000u) ? (k ^ 0x80000000u) : ~k;
    float s;
    __builtin_memcpy(&s, &u, 4);
    return s;
}
// 64-bit selection key: (score key, then lower row index first).  Row ids
// are below 2^31, so a real key is always above 0 (the padding key).
__host__ __device__ inline uint64_t pack_key(float s, uint32_t row) {
    return ((uint64_t)score_key(s) << 32) | (uint64_t)(0xFFFFFFFFu - row);
}
__host__ __device__ inline uint32_t key_row(uint64_t k) {
    return 0xFFFFFFFFu - (uint32_t)(k & 0xFFFFFFFFu);
}

// Round-to-nearest-even of a binary32 value into binary16 (dt = DT_F16) or
// bfloat16 bits; NaN stays a quiet NaN.  Exact for representable values.
__device__ inline uint16_t to_bits16(float f, int dt) {
    if (dt == DT_F16) {
        const _Float16 h = (_Float16)f;
        uint16_t b;
        __builtin_memcpy(&b, &h, 2);
        return b;
    }
    uint32_t u;
    __builtin_memcpy(&u, &f, 4);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// Bitonic sort of s[0..p) (LDS) into descending order by the kT threads of
// the block; p a power of two.  Every thread of the block must call it.
template <int kT>
__device__ inline void bitonic_desc(uint64_t* s, int p) {
    for (int size = 2; size <= p; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = threadIdx.x; i < (p >> 1); i += kT) {
                const int pos = 2 * i - (i & (stride - 1));
                const int partner = pos + stride;
                const bool desc = (pos & size) == 0;
                const uint64_t a = s[pos], b = s[partner];
                if ((a < b) == desc) {
                    s[pos] = b;
                    s[partner] = a;
                }
            }
            __syncthreads();
        }
    }
}

// ----------------------------------------------------------------- launchers
// Each returns hipSuccess or the launch error.  Shapes are validated by the
// caller (sense_api.hip) before these are reached.

// inv_norm[i] = 1 / ||keys[i, :d]|| (0 for a zero row), fp32 accumulation,
// when inv_norm is not NULL; the largest ||keys[i, :d]|| that is a number
// atomically maxed (as bits) into *max_norm_bits when that is not NULL.
hipError_t launch_key_norms(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                            float* inv_norm, uint32_t* max_norm_bits, hipStream_t stream);

// Query batches of at least this many run as an MFMA contraction, which
// reads the store once for the whole batch (a 16-query tile, padded); a
// single query runs the GEMV, whose fp32 query needs no hi/lo split.
constexpr int kMfmaMinQueries = 2;

// scores[q * n + i] = similarity of query q and row i for q in [0, nq).
// queries: nq x d fp32 (already converted).  inv_norm NULL for IP.  split:
// the queries are not exactly representable in the key type (MFMA path
// multiplies a hi and a lo half).  scratch: scan_scratch_bytes(nq, d) bytes.
hipError_t launch_scan(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                       const float* queries, int nq, bool split, const float* inv_norm,
                       float* scores, void* scratch, hipStream_t stream);
size_t scan_mfma_scratch_bytes(int nq, int d);
// One query group (<= 64 queries, already split) of the batched scan over
// rows 0, row_step, 2 row_step, ... (n_rows of them) of a store of row
// stride ld.  WRITE mode (scores != NULL): scores[q * n_rows + i].  FILTER
// mode (cand != NULL): rows whose score reaches the score of tau[q] go to
// query q's candidate list cand + q * cap as packed (score, row) keys: slots
// [w * kMfmaSlots, (w + 1) * kMfmaSlots) of wave w (the rest padding keys),
// then an overflow list whose next position is counts[q] (to be initialised
// to the slot area, mfma_scan_waves(n_rows) * kMfmaSlots).
struct MfmaScan {
    const void* keys;
    int key_dtype;
    int64_t ld;
    int64_t n_rows;
    int64_t row_step;
    int d;
    const uint16_t* qhi;
    const uint16_t* qlo;
    const float* inv_qn;
    int nq;
    const float* inv_norm;
    float* scores;            // WRITE mode
    const uint64_t* tau;      // FILTER mode
    int32_t* counts;
    uint64_t* cand;
    int64_t cap;
    const float* centre;      // PROJECT mode (proj_out set): out[key][o] =
    void* proj_out;           // (acc - centre[o]) * (normalize ? 1 / ||row|| : 1)
    int proj_dtype;
    int64_t proj_stride;
    int normalize;
    int proj_vec;             // 4 outputs per store (16-byte base, stride % 4, nq % 4)
};
constexpr int kMfmaSlots = 32;
hipError_t launch_scan_mfma_rows(const MfmaScan& s, bool split, hipStream_t stream);
int64_t mfma_scan_waves(int64_t n_rows);
hipError_t launch_scan_mfma(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                            const float* queries, int nq, bool split, const float* inv_norm,
                            float* scores, void* scratch, hipStream_t stream);

// Single-query scans of keys with d <= kSmallDim (several rows per load
// instruction), one launch per query.
hipError_t launch_scan_small(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                             const float* queries, int nq, const float* inv_norm, float* scores,
                             hipStream_t stream);

// PCA projection (+ L2 normalisation) of n rows; see project.hip.
bool project_uses_mfma(int x_dtype, const void* x, int64_t x_stride, int64_t n);
size_t project_workspace_bytes(int x_dtype, int64_t n, int d_in, int d_out);
// Fused projection of 16-bit rows onto at most kMfmaProjOut basis rows on the
// matrix cores: centring, normalisation and the store in the epilogue.
constexpr int kMfmaProjOut = 64;
hipError_t launch_project_mfma(const void* x, int x_dtype, int64_t n, int d_in, int64_t x_stride,
                               const float* basis, int d_out, const float* centre, int normalize,
                               void* out, int out_dtype, int64_t out_stride, void* scratch,
                               hipStream_t stream);
hipError_t launch_project(const void* x, int x_dtype, int64_t n, int d_in, int64_t x_stride,
                          const float* mean, const float* basis, int d_out, int normalize,
                          void* out, int out_dtype, int64_t out_stride, void* workspace,
                          hipStream_t stream);

// Top-k of packed keys (nq x count, padding key 0) in the order of the
// keys, with the gather; ids of padding keys are -1.  Query q has only its
// first dev_count[q] <= count keys (dev_count: nq counts on the device).  No
// workspace.
hipError_t launch_topk_keys(const uint64_t* keys, int64_t count, int nq, int k,
                            const int32_t* spans, const int32_t* span_len, int max_span,
                            int64_t span_stride, int64_t* out_ids, float* out_scores,
                            int32_t* out_drafts, int32_t* out_draft_len,
                            const int32_t* dev_count, hipStream_t stream);

// Inverted file (ivf.hip).
hipError_t launch_ivf_assign(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                             const float* centroids, int nlist, int cosine, int32_t* out_list,
                             hipStream_t stream);
hipError_t launch_pq_encode(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                            const float* centroids, int nlist, const int32_t* list_ids,
                            const float* codebooks, int m, int ksub, uint8_t* codes,
                            hipStream_t stream);
hipError_t launch_f32_inv_norms(const float* rows, int n, int d, float* inv, hipStream_t stream);
// Counting sort of the rows by list; counts has nlist + 2 entries (the last
// two count out-of-range list ids and codes).
hipError_t launch_ivf_layout(const int32_t* list_ids, int64_t n, int nlist, const void* keys,
                             int64_t ld, int d, const uint8_t* codes, int m, int ksub,
                             int32_t* counts, int64_t* offsets, int32_t* cursor,
                             int32_t* row_ids, void* keys_sorted, uint8_t* codes_sorted,
                             hipStream_t stream);

struct IvfSearch {
    const float* queries;      // nq x d fp32
    int d, nq;
    const float* centroids;    // nlist x d fp32
    const float* cen_inv;      // nlist (cosine)
    int nlist, cosine;
    float* coarse;             // nq x nlist
    float* coarse_ip;          // nq x nlist (PQ)
    int64_t* probe;            // nq x nprobe
    void* probe_ws;
    int nprobe;
    const int64_t* offsets;    // nlist + 1
    int32_t* count;            // nq: candidates of each query (sum of its probed list sizes)
    int64_t cap;               // candidate slots per query
    uint64_t* cand;            // nq x cap
    const uint8_t* codes_sorted;   // PQ, NULL for Flat
    int m, ksub;
    const float* codebooks;
    const void* keys_sorted;   // Flat
    int key_dtype;
    const float* inv_norm;     // Flat cosine, per sorted row
    const int32_t* row_ids;    // sorted position -> original row
    int k;
    const int32_t* spans;
    const int32_t* span_len;
    int max_span;
    int64_t span_stride;
    int64_t* out_ids;
    float* out_scores;
    int32_t* out_drafts;
    int32_t* out_draft_len;
};
hipError_t launch_ivf_search(const IvfSearch& s, hipStream_t stream);

// Compute units of the current device, queried once per process (every GPU
// this library drives is the same MI355X part).
int device_cus();

// Resident blocks of `kern` per compute unit at `threads` threads and no
// dynamic LDS, or `fallback` when the query fails; callers keep it in a
// function-local static (initialised once, also under concurrent calls).
template <typename Kernel>
int blocks_per_cu(Kernel kern, int threads, int fallback) {
    int v = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, kern, threads, 0) != hipSuccess || v < 1)
        v = fallback;
    return v;
}

// The queries of a batch padded to qpad = 16*ceil(nq/16) rows and split
// into hi + lo halves of the key type (a scratch of scan_mfma_scratch_bytes),
// with inv_qn[q] = 1/||q|| (cosine), 1 (inner product), 0 (padding), and
// margin[q]: twice a bound on |hi-only matrix-core score - fp32 rescore| of
// any row (cosine; inner product given the store's largest key norm; else 0).
struct QuerySplit {
    uint16_t* hi;
    uint16_t* lo;
    float* inv_qn;
    float* margin;
    int qpad;
};
QuerySplit query_split_parts(void* scratch, int nq, int d);
// key_norm_max (inner product, may be NULL): the store's largest key norm,
// which scales the inner-product margin.
hipError_t launch_query_split(const float* queries, int nq, int d, int key_dtype, bool cosine,
                              const float* key_norm_max, void* scratch, hipStream_t stream);

// Batched scan of short keys (d <= kSmallDim) on the matrix cores, for at
// most 64 queries of a split batch (see scan_short.hip).  Row r of the scan
// is stored row r * row_step.  WRITE: scores[q * n_rows + r].  FILTER: a row
// whose packed key (score, r * row_step) is at least tau[q] goes to
// cand[q * cap + ...]: wave w of short_scan_waves(n_rows) fills its slots
// [w * kShortSlots, (w + 1) * kShortSlots) (the rest padding keys), and the
// overflow is appended at counts[q] (which starts at the slot area's size).
constexpr int kShortSlots = 4;
int64_t short_scan_waves(int64_t n_rows);
struct ShortScan {
    const void* keys;
    int key_dtype;
    int64_t ld;
    int64_t n_rows;
    int64_t row_step;
    int d;
    const uint16_t* qhi;
    const uint16_t* qlo;
    const float* inv_qn;
    int nq;
    bool split;
    const float* inv_norm;
    float* scores;            // WRITE mode
    const uint64_t* tau;      // FILTER mode
    int32_t* counts;
    uint64_t* cand;
    int64_t cap;
};
hipError_t launch_scan_short(const ShortScan& s, hipStream_t stream);
// tau[q] = packed key of the k-th best row of a strided sample (the sample
// top-k's ids are sample positions; row = id * row_step), its score lowered
// by margin[q] when margin is not NULL; counts[q] = slot_area.
hipError_t launch_short_tau(const int64_t* ids, const float* scores, int nq, int k,
                            int64_t row_step, int32_t slot_area, const float* margin,
                            uint64_t* tau, int32_t* counts, hipStream_t stream);
// The band and rescore stages of a hi-only filtered search (scan_mfma.hip):
// launch_band keeps the candidates whose approximate score reaches
// kth[q * k + k - 1] - margin[q] (counts become the band sizes);
// launch_rescore replaces each band entry by its fp32 rescore.
hipError_t launch_band(uint64_t* cand, int64_t cap, int nq, const float* kth, int k,
                       const float* margin, int32_t* counts, hipStream_t stream);
hipError_t launch_rescore(uint64_t* cand, int64_t cap, int nq, const int32_t* counts,
                          const void* keys, int key_dtype, int64_t ld, int d,
                          const float* queries, const float* inv_norm, const float* inv_qn,
                          hipStream_t stream);

// Plain streaming read of a device buffer (bandwidth probe).
hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, hipStream_t stream);

// Converts nq x d queries of dtype q_dtype to fp32 (plain copy for fp32).
hipError_t launch_query_to_f32(const void* q, int q_dtype, int nq, int d, float* out,
                               hipStream_t stream);

// Workspace of the top-k stage, in bytes, for nq queries over n scores.
size_t topk_workspace_bytes(int64_t n, int nq, int k);

// Per-query top-k of scores (nq x n) in the order (score desc, row asc),
// plus the gather of each hit's continuation: row i's tokens start at
// spans[i * span_stride] (span_stride = max_span for a table of rows, 1 for
// a token history whose continuations overlap).
hipError_t launch_topk_gather(const float* scores, int64_t n, int nq, int k,
                              const int32_t* spans, const int32_t* span_len, int max_span,
                              int64_t span_stride, int64_t* out_ids, float* out_scores, int32_t* out_drafts,
                              int32_t* out_draft_len, void* workspace, hipStream_t stream);

// Verification workspace in bytes.
size_t verify_workspace_bytes(int n_cand, int max_len, int vocab);

struct GateParams {
    float gamma;
    int topk;
    int window;
    int tau;
    float ent_scale;  // 1/ln V when normalised, 1 otherwise
};

hipError_t launch_verify(const void* logits, int logits_dtype, int64_t row_stride,
                         const int32_t* drafts, const int32_t* draft_len, int n_cand,
                         int max_len, int vocab, int n_groups, const GateParams& gp,
                         int32_t* out_accept_len, int32_t* out_best, float* out_gate_score,
                         uint8_t* out_masks, int32_t* out_rank, void* workspace,
                         hipStream_t stream);

// Composite-score selection (one block per query); pool n_s + n_d <= kMaxPool.
struct SelectParams {
    float alpha;
    float beta;
    float delta;
    int anchor_override;
};

hipError_t launch_select_candidates(const float* scores_s, const int32_t* drafts_s,
                                    const int32_t* len_s, int n_s, const float* scores_d,
                                    const int32_t* drafts_d, const int32_t* len_d, int n_d,
                                    const int32_t* anchors, int n_queries, int max_len,
                                    int top_n, const SelectParams& sp, int32_t* out_drafts,
                                    int32_t* out_len, int32_t* out_source, float* out_score,
                                    hipStream_t stream);

// Appends `count` rows to a dynamic cache of n_old rows: keys (count x d of
// src_dtype, converted to key_dtype) into keys (row stride d), tokens into
// the history, the continuation lengths min(max_span, n - p), and, when
// inv_norm is not NULL, each new row's 1/||k|| (as the index build forms it);
// when max_norm_bits is not NULL, the new rows' norms maxed into it.
hipError_t launch_append_rows(const void* src, int src_dtype, int key_dtype,
                              const int32_t* tokens, int d, int64_t n_old, int count,
                              int max_span, void* keys, int32_t* hist, int32_t* span_len,
                              float* inv_norm, uint32_t* max_norm_bits, hipStream_t stream);

// Outputs of the loose-trie build (device pointers; NULL = not wanted for
// the optional ones).  Per group g of gs drafts of m tokens, nodes = gs * m
// entries of the per-node arrays start at g * nodes.
struct TrieOut {
    int32_t* order;          // n_cand: original index of each sorted draft
    int32_t* gamma;          // n_cand x m: tree id of each existing position, else -1
    int32_t* tokens;         // node tokens (-1 past L)
    int32_t* parent;         // node parent (-1 at depth 0 and past L)
    int32_t* depth;          // node depth (-1 past L)
    int32_t* cand;           // sorted draft creating the node (-1 past L)
    int32_t* tree_len;       // n_groups: L
    int32_t* sorted_drafts;  // optional n_cand x m (-1 padded)
    int32_t* sorted_len;     // optional n_cand
    uint8_t* mask;           // optional ancestor mask, nodes rows per group
    int64_t mask_ld;
    void* full_mask;         // optional static-KV mask, nodes rows x cache_len
    int full_dtype;
    int prefix_len;
    int64_t cache_len;
};

hipError_t launch_trie(const int32_t* drafts, const int32_t* draft_len, int n_cand, int max_len,
                       int n_groups, const TrieOut& out, hipStream_t stream);

// Verification through the tree: logits hold, per group, row 0 = the
// current position's distribution and row 1 + u = the distribution after
// tree node u; candidate c's token j is tree node gamma[c][j].
size_t verify_tree_workspace_bytes(int n_cand, int max_len, int vocab, int n_groups);
hipError_t launch_verify_tree(const void* logits, int logits_dtype, int64_t row_stride,
                              const int32_t* tree_tokens, const int32_t* tree_parent,
                              const int32_t* tree_len, const int32_t* gamma, int n_cand,
                              int max_len, int vocab, int n_groups, const GateParams& gp,
                              int32_t* out_accept_len, int32_t* out_best, float* out_gate_score,
                              uint8_t* out_masks, int32_t* out_rank, void* workspace,
                              hipStream_t stream);

}  // namespace sense
