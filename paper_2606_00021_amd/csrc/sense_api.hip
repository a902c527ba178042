// Host layer of the C ABI declared in include/sense.h: argument validation,
// workspace layout, index ownership, and the launch sequence of each entry
// point.  No C++ exception crosses the boundary; every failure returns a
// status and leaves a message for sense_last_error_message().
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>

#include "internal.h"
#include "sense.h"

#define SENSE_EXPORT extern "C" __attribute__((visibility("default")))

struct sense_index {
    const void* keys;       // borrowed or owned (== owned_keys)
    void* owned_keys;       // SENSE_INDEX_COPY_KEYS copy, else NULL
    int key_dtype;
    int64_t n;
    int32_t d;
    int64_t ld;
    const int32_t* spans;
    int32_t max_span;
    const int32_t* span_len;
    int64_t span_stride;    // elements between consecutive rows of `spans`
    int metric;
    float* inv_norm;        // owned; NULL for the inner-product metric
    uint32_t* key_norm_max; // owned, inner product only: the largest key norm (float bits)
    // Dynamic context cache only: capacity > 0, owned token history (the
    // span table, row stride 1) and continuation lengths.
    int64_t capacity;
    int32_t* owned_hist;
    int32_t* owned_span_len;
    // Inverted file only (nlist > 0).
    int32_t nlist;
    float* centroids;        // nlist x d
    float* cen_inv;          // nlist
    int32_t* counts;         // nlist + 2
    int32_t* cursor;         // nlist
    int64_t* offsets;        // nlist + 1
    int32_t* row_ids;        // n
    uint8_t* codes_sorted;   // n x pq_m (PQ)
    float* codebooks;        // pq_m x pq_ksub x d / pq_m (PQ)
    int32_t pq_m, pq_ksub;
    int64_t* cap_prefix;     // host: sums of the p largest list sizes, p = 0..nlist
};

namespace {

thread_local char g_msg[512];

// Timing events per sense_timer_t, set by sense_set_timer_events.
constexpr int kTimers = 8;
thread_local hipEvent_t g_timer[kTimers][2] = {};

hipError_t timer_mark(int which, int edge, hipStream_t st) {
    hipEvent_t ev = g_timer[which][edge];
    return ev ? hipEventRecord(ev, st) : hipSuccess;
}

sense_status_t fail(sense_status_t st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_msg, sizeof g_msg, fmt, ap);
    va_end(ap);
    return st;
}

sense_status_t ok() {
    g_msg[0] = '\0';
    return SENSE_OK;
}

sense_status_t hip_fail(hipError_t e, const char* where) {
    return fail(SENSE_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int elem_size(int dt) { return dt == SENSE_F32 ? 4 : 2; }

bool dtype_ok(int dt) { return dt == SENSE_F32 || dt == SENSE_F16 || dt == SENSE_BF16; }

// Retrieval workspace layout:
// [fp32 queries | split queries (MFMA path) | scores | top-k buffers].
struct RetrieveLayout {
    size_t q_off, m_off, s_off, t_off, total;
};

// Batched queries over short keys: the matrix-core short-key scan, with a
// sampled threshold and a filtered pass when the store is large.
constexpr int64_t kShortSample = 32768;      // rows of the threshold sample
constexpr int64_t kShortDirectMax = 131072;  // up to this many rows: plain scores + top-k

bool short_batched(const sense_index* ix, int nq) {
    return ix->d <= sense::kSmallDim && nq >= sense::kMfmaMinQueries;
}

// Long keys, query batches: the matrix-core scan.  Stores of more than
// kBatchDirectMax rows are searched like the short keys (a strided sample's
// k-th best as the threshold of a filtered pass), smaller ones through the
// plain score matrix.
constexpr int64_t kBatchSample = 32768;
constexpr int64_t kBatchDirectMax = 131072;

bool long_batched(const sense_index* ix, int nq) {
    return ix->d > sense::kSmallDim && nq >= sense::kMfmaMinQueries;
}

struct ShortLayout {
    size_t q_off, m_off, ss_off, sid_off, ssc_off, sws_off, tau_off, cnt_off, cand_off, fws_off,
        total;
    int64_t cap;    // entries of one query's candidate list
};

// Workspace of the sampled-threshold retrieval (short keys, or long keys in
// batches): query split, sample scores and top-k, thresholds and counts, the
// candidate lists (wave slots + an overflow list of up to every row) or, for
// a store searched directly, the plain score matrix in the same area.
ShortLayout short_layout(const sense_index* ix, int nq, int k) {
    ShortLayout l;
    const bool long_keys = ix->d > sense::kSmallDim;
    const int64_t sample = long_keys ? kBatchSample : kShortSample;
    const int64_t rows = ix->capacity > 0 ? ix->capacity : ix->n;
    const int g = nq < 64 ? nq : 64;
    size_t at = 0;
    auto take = [&](size_t bytes) {
        const size_t o = at;
        at = round_up(at + bytes, 256);
        return o;
    };
    l.q_off = take((size_t)nq * ix->d * sizeof(float));
    l.m_off = take(sense::scan_mfma_scratch_bytes(nq, ix->d));
    l.ss_off = take((size_t)g * sample * sizeof(float));
    l.sid_off = take((size_t)g * k * sizeof(int64_t));
    l.ssc_off = take((size_t)g * k * sizeof(float));
    l.sws_off = take(sense::topk_workspace_bytes(sample, g, k));
    l.tau_off = take((size_t)g * sizeof(uint64_t));
    l.cnt_off = take((size_t)g * sizeof(int32_t));
    // candidates per query: the wave slots, then an overflow list of up to
    // every row; also the plain score matrix of small stores
    const int64_t cap = long_keys ? sense::mfma_scan_waves(rows) * sense::kMfmaSlots + rows
                                  : sense::short_scan_waves(rows) * sense::kShortSlots + rows;
    l.cap = cap;
    l.cand_off = take((size_t)g * cap * sizeof(uint64_t));
    l.fws_off = take(sense::topk_workspace_bytes(cap, g, k));
    l.total = at;
    return l;
}

RetrieveLayout retrieve_layout(const sense_index* ix, int nq, int k) {
    RetrieveLayout l;
    if (short_batched(ix, nq) || long_batched(ix, nq)) {
        const ShortLayout sl = short_layout(ix, nq, k);
        l.q_off = sl.q_off;
        l.m_off = sl.m_off;
        l.s_off = sl.cand_off;
        l.t_off = sl.fws_off;
        l.total = sl.total;
        return l;
    }
    l.q_off = 0;
    l.m_off = round_up((size_t)nq * ix->d * sizeof(float), 256);
    const size_t mfma = nq >= sense::kMfmaMinQueries ? sense::scan_mfma_scratch_bytes(nq, ix->d) : 0;
    l.s_off = l.m_off + round_up(mfma, 256);
    // A dynamic cache is sized for its capacity, so one workspace serves
    // every later row count.
    const int64_t rows = ix->capacity > 0 ? ix->capacity : ix->n;
    l.t_off = l.s_off + round_up((size_t)nq * (size_t)rows * sizeof(float), 256);
    l.total = l.t_off + sense::topk_workspace_bytes(rows, nq, k);
    return l;
}

}  // namespace

SENSE_EXPORT const char* sense_status_string(sense_status_t s) {
    switch (s) {
        case SENSE_OK: return "ok";
        case SENSE_ERR_INVALID_ARGUMENT: return "invalid argument";
        case SENSE_ERR_MISALIGNED: return "misaligned pointer or stride";
        case SENSE_ERR_UNSUPPORTED: return "unsupported size";
        case SENSE_ERR_OUT_OF_MEMORY: return "out of device memory";
        case SENSE_ERR_WORKSPACE: return "workspace missing or too small";
        case SENSE_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

SENSE_EXPORT const char* sense_last_error_message(void) { return g_msg; }

SENSE_EXPORT sense_status_t sense_set_timer_events(sense_timer_t which, void* start_event,
                                                   void* stop_event) {
    if ((int)which < 0 || (int)which >= kTimers)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown timer %d", (int)which);
    if ((start_event == nullptr) != (stop_event == nullptr))
        return fail(SENSE_ERR_INVALID_ARGUMENT, "give both events or neither");
    g_timer[which][0] = (hipEvent_t)start_event;
    g_timer[which][1] = (hipEvent_t)stop_event;
    return ok();
}

SENSE_EXPORT sense_status_t sense_build_index(const sense_index_desc_t* desc, void* stream,
                                              sense_index_t** out) {
    if (!desc || !out) return fail(SENSE_ERR_INVALID_ARGUMENT, "desc and out must be non-NULL");
    *out = nullptr;
    const sense_index_desc_t& D = *desc;
    if (!D.keys || !D.spans) return fail(SENSE_ERR_INVALID_ARGUMENT, "keys and spans must be non-NULL");
    if (D.key_dtype != SENSE_F16 && D.key_dtype != SENSE_BF16)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "key_dtype must be SENSE_F16 or SENSE_BF16");
    if (D.n < 1 || D.n > 0x7FFFFFFFLL)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "n = %lld outside [1, 2^31-1]", (long long)D.n);
    if (D.d < 1 || D.d > sense::kMaxDim || D.d % 8 != 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "d = %d must be a multiple of 8 in [8, %d]", D.d,
                    sense::kMaxDim);
    if (D.key_stride < D.d)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "key_stride %lld < d %d", (long long)D.key_stride, D.d);
    if (D.max_span < 1 || D.max_span > sense::kMaxLen)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "max_span = %d outside [1, %d]", D.max_span,
                    sense::kMaxLen);
    if (D.metric != SENSE_METRIC_IP && D.metric != SENSE_METRIC_COSINE)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown metric %d", (int)D.metric);
    if ((D.flags & ~SENSE_INDEX_COPY_KEYS) != 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown flags 0x%x", D.flags);
    const bool copy = (D.flags & SENSE_INDEX_COPY_KEYS) != 0;
    if (!copy && (!aligned(D.keys, 16) || D.key_stride % 8 != 0))
        return fail(SENSE_ERR_MISALIGNED,
                    "keys must be 16-byte aligned with key_stride %% 8 == 0 "
                    "(or pass SENSE_INDEX_COPY_KEYS)");

    sense_index* ix = new (std::nothrow) sense_index();
    if (!ix) return fail(SENSE_ERR_OUT_OF_MEMORY, "host allocation failed");
    ix->key_dtype = D.key_dtype;
    ix->n = D.n;
    ix->d = D.d;
    ix->spans = D.spans;
    ix->max_span = D.max_span;
    ix->span_len = D.span_len;
    ix->span_stride = D.max_span;
    ix->metric = D.metric;
    hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    if (copy) {
        ix->ld = D.d;  // d % 8 == 0, so rows stay 16-byte aligned
        const size_t bytes = (size_t)D.n * D.d * 2;
        if ((e = hipMalloc(&ix->owned_keys, bytes)) != hipSuccess) {
            delete ix;
            return fail(SENSE_ERR_OUT_OF_MEMORY, "key copy of %zu bytes: %s", bytes,
                        hipGetErrorString(e));
        }
        e = hipMemcpy2DAsync(ix->owned_keys, (size_t)D.d * 2, D.keys, (size_t)D.key_stride * 2,
                             (size_t)D.d * 2, (size_t)D.n, hipMemcpyDeviceToDevice, st);
        if (e != hipSuccess) {
            (void)hipFree(ix->owned_keys);
            delete ix;
            return hip_fail(e, "key copy");
        }
        ix->keys = ix->owned_keys;
    } else {
        ix->keys = D.keys;
        ix->ld = D.key_stride;
    }
    // Cosine: the inverse-norm table.  Inner product: the largest key norm,
    // which bounds the error of the batched search's hi-only pass.
    const bool cos = D.metric == SENSE_METRIC_COSINE;
    e = cos ? hipMalloc(&ix->inv_norm, (size_t)D.n * sizeof(float))
            : hipMalloc((void**)&ix->key_norm_max, sizeof(uint32_t));
    if (e != hipSuccess) {
        if (ix->owned_keys) (void)hipFree(ix->owned_keys);
        delete ix;
        return fail(SENSE_ERR_OUT_OF_MEMORY, "norm table: %s", hipGetErrorString(e));
    }
    if (!cos) e = hipMemsetAsync(ix->key_norm_max, 0, sizeof(uint32_t), st);
    if (e == hipSuccess)
        e = sense::launch_key_norms(ix->keys, ix->key_dtype, ix->n, ix->d, ix->ld, ix->inv_norm,
                                    ix->key_norm_max, st);
    if (e != hipSuccess) {
        if (ix->inv_norm) (void)hipFree(ix->inv_norm);
        if (ix->key_norm_max) (void)hipFree(ix->key_norm_max);
        if (ix->owned_keys) (void)hipFree(ix->owned_keys);
        delete ix;
        return hip_fail(e, "key norms");
    }
    *out = ix;
    return ok();
}

SENSE_EXPORT sense_status_t sense_build_dynamic_index(const sense_dynamic_index_desc_t* desc,
                                                      sense_index_t** out) {
    if (!desc || !out) return fail(SENSE_ERR_INVALID_ARGUMENT, "desc and out must be non-NULL");
    *out = nullptr;
    const sense_dynamic_index_desc_t& D = *desc;
    if (D.key_dtype != SENSE_F16 && D.key_dtype != SENSE_BF16)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "key_dtype must be SENSE_F16 or SENSE_BF16");
    if (D.capacity < 1 || D.capacity > 0x7FFFFFFFLL)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "capacity = %lld outside [1, 2^31-1]",
                    (long long)D.capacity);
    if (D.d < 1 || D.d > sense::kMaxDim || D.d % 8 != 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "d = %d must be a multiple of 8 in [8, %d]", D.d,
                    sense::kMaxDim);
    if (D.max_span < 1 || D.max_span > sense::kMaxLen)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "max_span = %d outside [1, %d]", D.max_span,
                    sense::kMaxLen);
    if (D.metric != SENSE_METRIC_IP && D.metric != SENSE_METRIC_COSINE)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown metric %d", (int)D.metric);
    sense_index* ix = new (std::nothrow) sense_index();
    if (!ix) return fail(SENSE_ERR_OUT_OF_MEMORY, "host allocation failed");
    ix->key_dtype = D.key_dtype;
    ix->n = 0;
    ix->d = D.d;
    ix->ld = D.d;
    ix->max_span = D.max_span;
    ix->span_stride = 1;
    ix->metric = D.metric;
    ix->capacity = D.capacity;
    const size_t rows = (size_t)D.capacity;
    hipError_t e = hipMalloc(&ix->owned_keys, rows * D.d * 2);
    if (e == hipSuccess) e = hipMalloc((void**)&ix->owned_hist, rows * sizeof(int32_t));
    if (e == hipSuccess) e = hipMalloc((void**)&ix->owned_span_len, rows * sizeof(int32_t));
    if (e == hipSuccess && D.metric == SENSE_METRIC_COSINE)
        e = hipMalloc((void**)&ix->inv_norm, rows * sizeof(float));
    if (e == hipSuccess && D.metric != SENSE_METRIC_COSINE) {
        // zeroed by a synchronous copy: the cache's appends may come on any stream
        const uint32_t zero = 0;
        e = hipMalloc((void**)&ix->key_norm_max, sizeof(uint32_t));
        if (e == hipSuccess)
            e = hipMemcpy(ix->key_norm_max, &zero, sizeof(uint32_t), hipMemcpyHostToDevice);
    }
    if (e != hipSuccess) {
        if (ix->owned_keys) (void)hipFree(ix->owned_keys);
        if (ix->owned_hist) (void)hipFree(ix->owned_hist);
        if (ix->owned_span_len) (void)hipFree(ix->owned_span_len);
        if (ix->inv_norm) (void)hipFree(ix->inv_norm);
        if (ix->key_norm_max) (void)hipFree(ix->key_norm_max);
        delete ix;
        return fail(SENSE_ERR_OUT_OF_MEMORY, "dynamic cache of %lld rows: %s",
                    (long long)D.capacity, hipGetErrorString(e));
    }
    ix->keys = ix->owned_keys;
    ix->spans = ix->owned_hist;
    ix->span_len = ix->owned_span_len;
    *out = ix;
    return ok();
}

SENSE_EXPORT sense_status_t sense_index_append(sense_index_t* ix, const void* keys,
                                               sense_dtype_t keys_dtype, const int32_t* tokens,
                                               int32_t count, void* stream) {
    if (!ix) return fail(SENSE_ERR_INVALID_ARGUMENT, "index is NULL");
    if (ix->capacity == 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "index is not a dynamic cache");
    if (count < 0) return fail(SENSE_ERR_INVALID_ARGUMENT, "count = %d < 0", count);
    if (!dtype_ok(keys_dtype))
        return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown keys dtype %d", (int)keys_dtype);
    if (ix->n + count > ix->capacity)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "append of %d rows to %lld exceeds capacity %lld",
                    count, (long long)ix->n, (long long)ix->capacity);
    if (count == 0) return ok();
    if (!keys || !tokens) return fail(SENSE_ERR_INVALID_ARGUMENT, "keys and tokens must be non-NULL");
    if (!aligned(keys, (size_t)elem_size(keys_dtype)) || !aligned(tokens, 4))
        return fail(SENSE_ERR_MISALIGNED, "keys or tokens not aligned to their element size");
    hipStream_t st = (hipStream_t)stream;
    // The new rows' 1/||k|| (cosine) are formed by the same launch.
    hipError_t e = sense::launch_append_rows(keys, keys_dtype, ix->key_dtype, tokens, ix->d, ix->n,
                                             count, ix->max_span, ix->owned_keys, ix->owned_hist,
                                             ix->owned_span_len, ix->inv_norm, ix->key_norm_max,
                                             st);
    if (e != hipSuccess) return hip_fail(e, "append");
    ix->n += count;
    return ok();
}

SENSE_EXPORT sense_status_t sense_destroy_index(sense_index_t* ix) {
    if (!ix) return ok();
    hipError_t e = hipDeviceSynchronize();
    if (ix->inv_norm) (void)hipFree(ix->inv_norm);
    if (ix->key_norm_max) (void)hipFree(ix->key_norm_max);
    if (ix->owned_keys) (void)hipFree(ix->owned_keys);
    if (ix->owned_hist) (void)hipFree(ix->owned_hist);
    if (ix->owned_span_len) (void)hipFree(ix->owned_span_len);
    for (void* p : {(void*)ix->centroids, (void*)ix->cen_inv, (void*)ix->counts,
                    (void*)ix->cursor, (void*)ix->offsets, (void*)ix->row_ids,
                    (void*)ix->codes_sorted, (void*)ix->codebooks})
        if (p) (void)hipFree(p);
    delete[] ix->cap_prefix;
    delete ix;
    if (e != hipSuccess) return hip_fail(e, "destroy");
    return ok();
}

SENSE_EXPORT sense_status_t sense_index_info(const sense_index_t* ix, int64_t* n, int32_t* d,
                                             int32_t* max_span, sense_metric_t* metric,
                                             sense_dtype_t* key_dtype) {
    if (!ix) return fail(SENSE_ERR_INVALID_ARGUMENT, "index is NULL");
    if (n) *n = ix->n;
    if (d) *d = ix->d;
    if (max_span) *max_span = ix->max_span;
    if (metric) *metric = (sense_metric_t)ix->metric;
    if (key_dtype) *key_dtype = (sense_dtype_t)ix->key_dtype;
    return ok();
}

static sense_status_t check_retrieve_sizes(const sense_index_t* ix, int32_t nq, int32_t k) {
    if (!ix) return fail(SENSE_ERR_INVALID_ARGUMENT, "index is NULL");
    if (ix->nlist > 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT,
                    "an inverted-file index is searched with sense_ivf_search");
    if (nq < 1) return fail(SENSE_ERR_INVALID_ARGUMENT, "n_queries = %d < 1", nq);
    if (k < 1) return fail(SENSE_ERR_INVALID_ARGUMENT, "k = %d < 1", k);
    if (k > sense::kMaxK) return fail(SENSE_ERR_UNSUPPORTED, "k = %d > %d", k, sense::kMaxK);
    if ((int64_t)k > ix->n)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "k = %d exceeds the %lld stored rows", k,
                    (long long)ix->n);
    // Batches keep per-query candidate lists (wave slots, then up to every
    // row) whose positions are 32-bit.
    if (short_batched(ix, nq) || long_batched(ix, nq)) {
        const ShortLayout L = short_layout(ix, nq, k);
        if (L.cap > (int64_t)INT32_MAX)
            return fail(SENSE_ERR_UNSUPPORTED,
                        "a batch over %lld rows needs candidate lists of %lld entries (at most "
                        "2^31 - 1): search it one query at a time",
                        (long long)(ix->capacity > 0 ? ix->capacity : ix->n), (long long)L.cap);
    }
    return SENSE_OK;
}

SENSE_EXPORT sense_status_t sense_retrieve_workspace_size(const sense_index_t* ix, int32_t nq,
                                                          int32_t k, size_t* bytes) {
    if (!bytes) return fail(SENSE_ERR_INVALID_ARGUMENT, "bytes is NULL");
    const sense_status_t s = check_retrieve_sizes(ix, nq, k);
    if (s != SENSE_OK) return s;
    *bytes = retrieve_layout(ix, nq, k).total;
    return ok();
}

// Short keys, query batch: per group of <= 64 queries either plain scores +
// top-k (small stores) or a strided sample's k-th best key as a threshold,
// a filtered pass over every row, and the top-k of the survivors.
static hipError_t retrieve_short(const sense_index* ix, const float* qptr, int nq, int k,
                                 bool split, int64_t* out_ids, float* out_scores,
                                 int32_t* out_drafts, int32_t* out_draft_len, char* ws,
                                 hipStream_t st) {
    const ShortLayout L = short_layout(ix, nq, k);
    const int64_t n = ix->n;
    hipError_t e;
    if ((e = timer_mark(SENSE_TIMER_SCAN, 0, st)) != hipSuccess) return e;
    if ((e = sense::launch_query_split(qptr, nq, ix->d, ix->key_dtype, ix->inv_norm != nullptr,
                                       nullptr, ws + L.m_off, st)) != hipSuccess)
        return e;
    const sense::QuerySplit qs = sense::query_split_parts(ws + L.m_off, nq, ix->d);
    const bool sample = n > kShortDirectMax;
    const int64_t step = sample ? n / kShortSample : 1;
    for (int g0 = 0; g0 < nq; g0 += 64) {
        const int ng = nq - g0 < 64 ? nq - g0 : 64;
        sense::ShortScan S{};
        S.keys = ix->keys;
        S.key_dtype = ix->key_dtype;
        S.ld = ix->ld;
        S.d = ix->d;
        S.qhi = qs.hi + (int64_t)g0 * ix->d;
        S.qlo = qs.lo + (int64_t)g0 * ix->d;
        S.inv_qn = qs.inv_qn + g0;
        S.nq = ng;
        S.split = split;
        S.inv_norm = ix->inv_norm;
        int64_t* gid = out_ids + (int64_t)g0 * k;
        float* gsc = out_scores ? out_scores + (int64_t)g0 * k : nullptr;
        int32_t* gdr = out_drafts ? out_drafts + (int64_t)g0 * k * ix->max_span : nullptr;
        int32_t* gdl = out_draft_len ? out_draft_len + (int64_t)g0 * k : nullptr;
        if (!sample) {
            S.n_rows = n;
            S.row_step = 1;
            S.scores = (float*)(ws + L.cand_off);
            if ((e = sense::launch_scan_short(S, st)) != hipSuccess) return e;
            if ((e = sense::launch_topk_gather(S.scores, n, ng, k, ix->spans, ix->span_len,
                                               ix->max_span, ix->span_stride, gid, gsc, gdr,
                                               gdl, ws + L.fws_off, st)) != hipSuccess)
                return e;
            continue;
        }
        // Threshold from the sample rows 0, step, 2 step, ...
        S.n_rows = kShortSample;
        S.row_step = step;
        S.scores = (float*)(ws + L.ss_off);
        if ((e = sense::launch_scan_short(S, st)) != hipSuccess) return e;
        int64_t* sid = (int64_t*)(ws + L.sid_off);
        float* ssc = (float*)(ws + L.ssc_off);
        if ((e = sense::launch_topk_gather(S.scores, kShortSample, ng, k, nullptr, nullptr, 1, 1,
                                           sid, ssc, nullptr, nullptr, ws + L.sws_off, st)) !=
            hipSuccess)
            return e;
        uint64_t* tau = (uint64_t*)(ws + L.tau_off);
        int32_t* cnt = (int32_t*)(ws + L.cnt_off);
        const int64_t slot_area = sense::short_scan_waves(n) * sense::kShortSlots;
        if ((e = sense::launch_short_tau(sid, ssc, ng, k, step, (int32_t)slot_area, nullptr,
                                         tau, cnt, st)) != hipSuccess)
            return e;
        // Every row; only keys >= tau are kept.
        S.n_rows = n;
        S.row_step = 1;
        S.scores = nullptr;
        S.tau = tau;
        S.counts = cnt;
        S.cand = (uint64_t*)(ws + L.cand_off);
        S.cap = slot_area + n;
        if ((e = sense::launch_scan_short(S, st)) != hipSuccess) return e;
        if ((e = sense::launch_topk_keys(S.cand, S.cap, ng, k, ix->spans, ix->span_len,
                                         ix->max_span, ix->span_stride, gid, gsc, gdr, gdl, cnt,
                                         st)) != hipSuccess)
            return e;
    }
    return timer_mark(SENSE_TIMER_SCAN, 1, st);
}

// Long keys, query batch: per group of <= 64 queries either plain scores +
// top-k (stores of up to kBatchDirectMax rows) or a strided sample's k-th
// best key as a threshold, a filtered matrix-core pass over every row, and
// the top-k of the survivors (exact: every row of the true top k reaches the
// threshold).
//
// A sampled threshold runs the matrix cores on the hi half of the query
// alone (half the instructions and query fragments of the hi + lo split;
// the split measured 1.3x slower at 64 queries) and makes up for it
// exactly: with b a bound on |approximate score A - fp32 rescore R| of any
// row (margin = 2b, per query; for inner product through the store's
// largest key norm),
//   threshold  = (sample's k-th best A) - 2b: the k sample rows reaching it
//                have R >= that + b, so the k-th best R is at least that + b
//                and every row of the R-top-k has A >= it;
//   band       = survivors with A >= (k-th best A of the survivors) - 2b:
//                the same argument over the survivors, which hold the A-top-k;
//   rescore    = R of every band row (fp32, as the single-query scan);
//   result     = the top k of the band by (R desc, row asc).
//
// Timers: SCAN spans the query split, the sample, its top-k and the filtered
// pass; FILTER the first query group's filtered pass alone; TOPK the rest.
static hipError_t retrieve_batched(const sense_index* ix, const float* qptr, int nq, int k,
                                   bool split, int64_t* out_ids, float* out_scores,
                                   int32_t* out_drafts, int32_t* out_draft_len, char* ws,
                                   hipStream_t st) {
    const ShortLayout L = short_layout(ix, nq, k);
    const int64_t n = ix->n;
    hipError_t e;
    if ((e = timer_mark(SENSE_TIMER_SCAN, 0, st)) != hipSuccess) return e;
    if ((e = sense::launch_query_split(qptr, nq, ix->d, ix->key_dtype, ix->inv_norm != nullptr,
                                       (const float*)ix->key_norm_max, ws + L.m_off, st)) !=
        hipSuccess)
        return e;
    const sense::QuerySplit qs = sense::query_split_parts(ws + L.m_off, nq, ix->d);
    const bool sample = n > kBatchDirectMax;
    const bool rescore = sample;
    const bool mfma_split = split && !rescore;
    const int64_t step = sample ? n / kBatchSample : 1;
    const int64_t slot_area = sense::mfma_scan_waves(n) * sense::kMfmaSlots;
    for (int g0 = 0; g0 < nq; g0 += 64) {
        const int ng = nq - g0 < 64 ? nq - g0 : 64;
        sense::MfmaScan S{};
        S.keys = ix->keys;
        S.key_dtype = ix->key_dtype;
        S.ld = ix->ld;
        S.d = ix->d;
        S.qhi = qs.hi + (int64_t)g0 * ix->d;
        S.qlo = qs.lo + (int64_t)g0 * ix->d;
        S.inv_qn = qs.inv_qn + g0;
        S.nq = ng;
        S.inv_norm = ix->inv_norm;
        int64_t* gid = out_ids + (int64_t)g0 * k;
        float* gsc = out_scores ? out_scores + (int64_t)g0 * k : nullptr;
        int32_t* gdr = out_drafts ? out_drafts + (int64_t)g0 * k * ix->max_span : nullptr;
        int32_t* gdl = out_draft_len ? out_draft_len + (int64_t)g0 * k : nullptr;
        const bool first = g0 == 0, last = g0 + 64 >= nq;
        if (!sample) {
            S.n_rows = n;
            S.row_step = 1;
            S.scores = (float*)(ws + L.cand_off);
            if ((e = sense::launch_scan_mfma_rows(S, mfma_split, st)) != hipSuccess) return e;
            if (last && (e = timer_mark(SENSE_TIMER_SCAN, 1, st)) != hipSuccess) return e;
            if (last && (e = timer_mark(SENSE_TIMER_TOPK, 0, st)) != hipSuccess) return e;
            if ((e = sense::launch_topk_gather(S.scores, n, ng, k, ix->spans, ix->span_len,
                                               ix->max_span, ix->span_stride, gid, gsc, gdr,
                                               gdl, ws + L.fws_off, st)) != hipSuccess)
                return e;
            continue;
        }
        // Threshold from the sample rows 0, step, 2 step, ...
        S.n_rows = kBatchSample;
        S.row_step = step;
        S.scores = (float*)(ws + L.ss_off);
        if ((e = sense::launch_scan_mfma_rows(S, mfma_split, st)) != hipSuccess) return e;
        int64_t* sid = (int64_t*)(ws + L.sid_off);
        float* ssc = (float*)(ws + L.ssc_off);
        if ((e = sense::launch_topk_gather(S.scores, kBatchSample, ng, k, nullptr, nullptr, 1, 1,
                                           sid, ssc, nullptr, nullptr, ws + L.sws_off, st)) !=
            hipSuccess)
            return e;
        uint64_t* tau = (uint64_t*)(ws + L.tau_off);
        int32_t* cnt = (int32_t*)(ws + L.cnt_off);
        const float* margin = rescore ? qs.margin + g0 : nullptr;
        if ((e = sense::launch_short_tau(sid, ssc, ng, k, step, (int32_t)slot_area, margin, tau,
                                         cnt, st)) != hipSuccess)
            return e;
        // Every row; only keys whose score reaches tau's are kept.
        S.n_rows = n;
        S.row_step = 1;
        S.scores = nullptr;
        S.tau = tau;
        S.counts = cnt;
        S.cand = (uint64_t*)(ws + L.cand_off);
        S.cap = slot_area + n;
        if (first && (e = timer_mark(SENSE_TIMER_FILTER, 0, st)) != hipSuccess) return e;
        if ((e = sense::launch_scan_mfma_rows(S, mfma_split, st)) != hipSuccess) return e;
        if (first && (e = timer_mark(SENSE_TIMER_FILTER, 1, st)) != hipSuccess) return e;
        if (last && (e = timer_mark(SENSE_TIMER_SCAN, 1, st)) != hipSuccess) return e;
        if (last && (e = timer_mark(SENSE_TIMER_TOPK, 0, st)) != hipSuccess) return e;
        if (rescore) {
            // k-th best approximate score of the survivors, the band, R.
            if ((e = sense::launch_topk_keys(S.cand, S.cap, ng, k, nullptr, nullptr, 1, 1, sid,
                                             ssc, nullptr, nullptr, cnt, st)) != hipSuccess)
                return e;
            if ((e = sense::launch_band(S.cand, S.cap, ng, ssc, k, margin, cnt, st)) !=
                hipSuccess)
                return e;
            if ((e = sense::launch_rescore(S.cand, S.cap, ng, cnt, ix->keys, ix->key_dtype,
                                           ix->ld, ix->d, qptr + (int64_t)g0 * ix->d,
                                           ix->inv_norm, S.inv_qn, st)) != hipSuccess)
                return e;
        }
        if ((e = sense::launch_topk_keys(S.cand, S.cap, ng, k, ix->spans, ix->span_len,
                                         ix->max_span, ix->span_stride, gid, gsc, gdr, gdl, cnt,
                                         st)) != hipSuccess)
            return e;
    }
    return timer_mark(SENSE_TIMER_TOPK, 1, st);
}

SENSE_EXPORT sense_status_t sense_retrieve(const sense_index_t* ix, const void* queries,
                                           sense_dtype_t q_dtype, int32_t nq, int32_t k,
                                           int64_t* out_ids, float* out_scores,
                                           int32_t* out_drafts, int32_t* out_draft_len,
                                           void* workspace, size_t workspace_bytes,
                                           void* stream) {
    sense_status_t s = check_retrieve_sizes(ix, nq, k);
    if (s != SENSE_OK) return s;
    if (!queries || !out_ids)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "queries and out_ids must be non-NULL");
    if (!dtype_ok(q_dtype)) return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown q_dtype %d", (int)q_dtype);
    if (!aligned(queries, q_dtype == SENSE_F32 ? 16 : 2))
        return fail(SENSE_ERR_MISALIGNED, "fp32 queries must be 16-byte aligned");
    const RetrieveLayout L = retrieve_layout(ix, nq, k);
    if (!workspace || workspace_bytes < L.total)
        return fail(SENSE_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", L.total,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 256)) return fail(SENSE_ERR_MISALIGNED, "workspace must be 256-byte aligned");

    hipStream_t st = (hipStream_t)stream;
    char* ws = (char*)workspace;
    float* qf = (float*)(ws + L.q_off);
    float* scores = (float*)(ws + L.s_off);
    hipError_t e;
    const float* qptr = (const float*)queries;
    if (q_dtype != SENSE_F32) {
        if ((e = sense::launch_query_to_f32(queries, q_dtype, nq, ix->d, qf, st)) != hipSuccess)
            return hip_fail(e, "query conversion");
        qptr = qf;
    }
    const bool split = q_dtype != ix->key_dtype;  // key-typed queries need no lo half
    if (short_batched(ix, nq)) {
        if ((e = retrieve_short(ix, qptr, nq, k, split, out_ids, out_scores, out_drafts,
                                out_draft_len, ws, st)) != hipSuccess)
            return hip_fail(e, "short-key batched retrieval");
        return ok();
    }
    if (long_batched(ix, nq)) {
        if ((e = retrieve_batched(ix, qptr, nq, k, split, out_ids, out_scores, out_drafts,
                                  out_draft_len, ws, st)) != hipSuccess)
            return hip_fail(e, "batched retrieval");
        return ok();
    }
    if ((e = timer_mark(SENSE_TIMER_SCAN, 0, st)) != hipSuccess) return hip_fail(e, "timer");
    if (ix->d <= sense::kSmallDim && nq < sense::kMfmaMinQueries)
        e = sense::launch_scan_small(ix->keys, ix->key_dtype, ix->n, ix->d, ix->ld, qptr, nq,
                                     ix->inv_norm, scores, st);
    else
        e = sense::launch_scan(ix->keys, ix->key_dtype, ix->n, ix->d, ix->ld, qptr, nq, split,
                               ix->inv_norm, scores, ws + L.m_off, st);
    if (e != hipSuccess) return hip_fail(e, "similarity scan");
    if ((e = timer_mark(SENSE_TIMER_SCAN, 1, st)) != hipSuccess) return hip_fail(e, "timer");
    if ((e = timer_mark(SENSE_TIMER_TOPK, 0, st)) != hipSuccess) return hip_fail(e, "timer");
    if ((e = sense::launch_topk_gather(scores, ix->n, nq, k, ix->spans, ix->span_len,
                                       ix->max_span, ix->span_stride, out_ids, out_scores, out_drafts,
                                       out_draft_len, ws + L.t_off, st)) != hipSuccess)
        return hip_fail(e, "top-k");
    if ((e = timer_mark(SENSE_TIMER_TOPK, 1, st)) != hipSuccess) return hip_fail(e, "timer");
    return ok();
}

// ---------------------------------------------------------------- retrieval
// without a caller workspace.  The scratch lives in this file-scope device
// array; every GPU the library runs on holds its own copy until the process
// ends.  In host code the array's name is only a stand-in for the symbol: the
// device address of each GPU's copy comes from hipGetSymbolAddress, taken
// once per device with that device current, and only that address is ever
// handed to a kernel.
static constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
void* g_scratch_ptr[kMaxScratchDevices];
hipError_t g_scratch_err[kMaxScratchDevices];
std::once_flag g_scratch_once[kMaxScratchDevices];
}  // namespace

static sense_status_t scratch_of_current_device(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxScratchDevices)
        return fail(SENSE_ERR_UNSUPPORTED, "device %d beyond the %d the static scratch serves",
                    dev, kMaxScratchDevices);
    std::call_once(g_scratch_once[dev], [dev] {
        g_scratch_err[dev] = hipGetSymbolAddress(&g_scratch_ptr[dev], HIP_SYMBOL(scratch));
    });
    if (g_scratch_err[dev] != hipSuccess) return hip_fail(g_scratch_err[dev], "hipGetSymbolAddress");
    if (!g_scratch_ptr[dev] || !aligned(g_scratch_ptr[dev], 256))
        return fail(SENSE_ERR_HIP, "static scratch of device %d has no usable address", dev);
    *out = g_scratch_ptr[dev];
    return SENSE_OK;
}

SENSE_EXPORT sense_status_t sense_retrieve_noalloc(const sense_index_t* ix, const void* queries,
                                                   sense_dtype_t q_dtype, int32_t nq, int32_t k,
                                                   int64_t* out_ids, float* out_scores,
                                                   int32_t* out_drafts, int32_t* out_draft_len,
                                                   void* stream) {
    sense_status_t s = check_retrieve_sizes(ix, nq, k);
    if (s != SENSE_OK) return s;
    const size_t need = retrieve_layout(ix, nq, k).total;
    if (need > kNoAllocScratchBytes)
        return fail(SENSE_ERR_UNSUPPORTED,
                    "this retrieval needs %zu bytes of scratch; the static scratch holds %zu "
                    "(call sense_retrieve with a workspace)", need, kNoAllocScratchBytes);
    void* ws = nullptr;
    if ((s = scratch_of_current_device(&ws)) != SENSE_OK) return s;
    return sense_retrieve(ix, queries, q_dtype, nq, k, out_ids, out_scores, out_drafts,
                          out_draft_len, ws, kNoAllocScratchBytes, stream);
}

SENSE_EXPORT size_t sense_retrieve_noalloc_max_bytes(void) { return kNoAllocScratchBytes; }

static sense_status_t check_verify_sizes(int32_t n_cand, int32_t max_len, int32_t vocab) {
    if (n_cand < 0) return fail(SENSE_ERR_INVALID_ARGUMENT, "n_cand = %d < 0", n_cand);
    if (max_len < 1 || max_len > sense::kMaxLen)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "max_len = %d outside [1, %d]", max_len,
                    sense::kMaxLen);
    if (vocab < 1) return fail(SENSE_ERR_INVALID_ARGUMENT, "vocab = %d < 1", vocab);
    if ((int64_t)n_cand * max_len > sense::kMaxVerifyRows)
        return fail(SENSE_ERR_UNSUPPORTED,
                    "n_cand * max_len = %lld rows; one call judges at most %lld (one block of "
                    "%d threads per row, under 2^32 work-items per dispatch)",
                    (long long)n_cand * max_len, (long long)sense::kMaxVerifyRows,
                    sense::kVerifyRowThreads);
    return SENSE_OK;
}

static sense_status_t check_gate_params(const sense_gate_params_t* params, int32_t vocab,
                                        sense::GateParams* gp) {
    if (!params) return fail(SENSE_ERR_INVALID_ARGUMENT, "params is NULL");
    if (params->topk < 1) return fail(SENSE_ERR_INVALID_ARGUMENT, "topk = %d < 1", params->topk);
    if (params->window < 0 || params->window > sense::kMaxLen)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "window = %d outside [0, %d]", params->window,
                    sense::kMaxLen);
    if (params->tau < 0) return fail(SENSE_ERR_INVALID_ARGUMENT, "tau = %d < 0", params->tau);
    if (params->gamma != params->gamma) return fail(SENSE_ERR_INVALID_ARGUMENT, "gamma is NaN");
    gp->gamma = params->gamma;
    gp->topk = params->topk;
    gp->window = params->window;
    gp->tau = params->tau;
    gp->ent_scale = params->entropy_normalized ? (float)(1.0 / log((double)vocab)) : 1.0f;
    if (vocab == 1) gp->ent_scale = params->entropy_normalized ? 0.0f : 1.0f;  // E = 0 = ln 1
    return SENSE_OK;
}

SENSE_EXPORT sense_status_t sense_soft_gate_verify_workspace_size(int32_t n_cand,
                                                                  int32_t max_len,
                                                                  int32_t vocab,
                                                                  size_t* bytes) {
    if (!bytes) return fail(SENSE_ERR_INVALID_ARGUMENT, "bytes is NULL");
    const sense_status_t s = check_verify_sizes(n_cand, max_len, vocab);
    if (s != SENSE_OK) return s;
    *bytes = sense::verify_workspace_bytes(n_cand, max_len, vocab);
    return ok();
}

SENSE_EXPORT sense_status_t sense_soft_gate_verify(
    const void* logits, sense_dtype_t logits_dtype, int64_t row_stride, const int32_t* drafts,
    const int32_t* draft_len, int32_t n_cand, int32_t max_len, int32_t vocab, int32_t n_groups,
    const sense_gate_params_t* params, int32_t* out_accept_len, int32_t* out_best,
    float* out_gate_score, uint8_t* out_masks, int32_t* out_rank, void* workspace,
    size_t workspace_bytes, void* stream) {
    sense_status_t s = check_verify_sizes(n_cand, max_len, vocab);
    if (s != SENSE_OK) return s;
    if (!params) return fail(SENSE_ERR_INVALID_ARGUMENT, "params is NULL");
    if (!dtype_ok(logits_dtype))
        return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown logits dtype %d", (int)logits_dtype);
    if (row_stride < vocab)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "row_stride %lld < vocab %d", (long long)row_stride, vocab);
    sense::GateParams gp;
    if ((s = check_gate_params(params, vocab, &gp)) != SENSE_OK) return s;
    if (n_cand == 0) return ok();
    if (n_groups < 1 || n_cand % n_groups != 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "n_groups = %d must divide n_cand = %d", n_groups,
                    n_cand);
    if (!logits || !drafts || !out_accept_len || !out_best)
        return fail(SENSE_ERR_INVALID_ARGUMENT,
                    "logits, drafts, out_accept_len and out_best must be non-NULL");
    if (!aligned(logits, (size_t)elem_size(logits_dtype)))
        return fail(SENSE_ERR_MISALIGNED, "logits not aligned to their element size");
    const size_t need = sense::verify_workspace_bytes(n_cand, max_len, vocab);
    if (!workspace || workspace_bytes < need)
        return fail(SENSE_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 256)) return fail(SENSE_ERR_MISALIGNED, "workspace must be 256-byte aligned");

    hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    if ((e = timer_mark(SENSE_TIMER_VERIFY, 0, st)) != hipSuccess) return hip_fail(e, "timer");
    e = sense::launch_verify(logits, logits_dtype, row_stride, drafts, draft_len, n_cand, max_len,
                             vocab, n_groups, gp, out_accept_len, out_best, out_gate_score,
                             out_masks, out_rank, workspace, st);
    if (e != hipSuccess) return hip_fail(e, "soft-gated evaluation");
    if ((e = timer_mark(SENSE_TIMER_VERIFY, 1, st)) != hipSuccess) return hip_fail(e, "timer");
    return ok();
}

SENSE_EXPORT sense_status_t sense_read_bandwidth_probe(const void* buf, size_t bytes,
                                                       uint32_t* sink, void* stream) {
    if (!buf || !sink || bytes == 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "buf and sink must be non-NULL, bytes > 0");
    if (!aligned(buf, 16) || bytes % 16 != 0)
        return fail(SENSE_ERR_MISALIGNED, "buf must be 16-byte aligned and bytes a multiple of 16");
    const hipError_t e = sense::launch_stream_read(buf, bytes, sink, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "read probe");
    return ok();
}

SENSE_EXPORT sense_status_t sense_select_candidates(
    const float* static_scores, const int32_t* static_drafts, const int32_t* static_len,
    int32_t n_static, const float* dynamic_scores, const int32_t* dynamic_drafts,
    const int32_t* dynamic_len, int32_t n_dynamic, const int32_t* anchors, int32_t n_queries,
    int32_t max_len, int32_t top_n, const sense_select_params_t* params, int32_t* out_drafts,
    int32_t* out_len, int32_t* out_source, float* out_score, void* stream) {
    if (!params) return fail(SENSE_ERR_INVALID_ARGUMENT, "params is NULL");
    if (n_static < 0 || n_dynamic < 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "n_static = %d and n_dynamic = %d must be >= 0",
                    n_static, n_dynamic);
    const int64_t pool = (int64_t)n_static + n_dynamic;
    if (pool < 1) return fail(SENSE_ERR_INVALID_ARGUMENT, "empty candidate pool");
    if (pool > sense::kMaxPool)
        return fail(SENSE_ERR_UNSUPPORTED, "pool of %lld candidates > %d", (long long)pool,
                    sense::kMaxPool);
    if (top_n < 1 || top_n > pool)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "top_n = %d outside [1, %lld]", top_n,
                    (long long)pool);
    if (max_len < 1 || max_len > sense::kMaxLen)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "max_len = %d outside [1, %d]", max_len,
                    sense::kMaxLen);
    if (n_queries < 1) return fail(SENSE_ERR_INVALID_ARGUMENT, "n_queries = %d < 1", n_queries);
    if (n_static > 0 && (!static_scores || !static_drafts))
        return fail(SENSE_ERR_INVALID_ARGUMENT, "static_scores and static_drafts must be non-NULL");
    if (n_dynamic > 0 && (!dynamic_scores || !dynamic_drafts))
        return fail(SENSE_ERR_INVALID_ARGUMENT,
                    "dynamic_scores and dynamic_drafts must be non-NULL");
    if (!anchors || !out_drafts || !out_len)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "anchors, out_drafts and out_len must be non-NULL");
    const sense_select_params_t& P = *params;
    if (P.alpha != P.alpha || P.beta != P.beta || P.delta != P.delta)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "alpha, beta and delta must not be NaN");
    const sense::SelectParams sp{P.alpha, P.beta, P.delta, P.anchor_override != 0};
    hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    if ((e = timer_mark(SENSE_TIMER_SELECT, 0, st)) != hipSuccess) return hip_fail(e, "timer");
    e = sense::launch_select_candidates(static_scores, static_drafts, static_len, n_static,
                                        dynamic_scores, dynamic_drafts, dynamic_len, n_dynamic,
                                        anchors, n_queries, max_len, top_n, sp, out_drafts,
                                        out_len, out_source, out_score, st);
    if (e != hipSuccess) return hip_fail(e, "candidate selection");
    if ((e = timer_mark(SENSE_TIMER_SELECT, 1, st)) != hipSuccess) return hip_fail(e, "timer");
    return ok();
}

static sense_status_t check_groups(int32_t n_cand, int32_t max_len, int32_t n_groups) {
    if (n_groups < 1 || n_cand % n_groups != 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "n_groups = %d must divide n_cand = %d", n_groups,
                    n_cand);
    const int gs = n_cand / n_groups;
    if (gs > sense::kMaxGroup || (int64_t)gs * max_len > sense::kMaxNodes)
        return fail(SENSE_ERR_UNSUPPORTED,
                    "group of %d drafts x %d tokens exceeds %d drafts or %d tokens", gs, max_len,
                    sense::kMaxGroup, sense::kMaxNodes);
    return SENSE_OK;
}

SENSE_EXPORT sense_status_t sense_build_loose_trie(const int32_t* drafts, const int32_t* draft_len,
                                                   int32_t n_cand, int32_t max_len,
                                                   int32_t n_groups, const sense_trie_t* out,
                                                   void* stream) {
    if (!out) return fail(SENSE_ERR_INVALID_ARGUMENT, "out is NULL");
    if (n_cand < 1) return fail(SENSE_ERR_INVALID_ARGUMENT, "n_cand = %d < 1", n_cand);
    if (max_len < 1 || max_len > sense::kMaxLen)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "max_len = %d outside [1, %d]", max_len,
                    sense::kMaxLen);
    sense_status_t s = check_groups(n_cand, max_len, n_groups);
    if (s != SENSE_OK) return s;
    const sense_trie_t& O = *out;
    if (!drafts || !O.order || !O.gamma || !O.tree_tokens || !O.tree_parent || !O.tree_depth ||
        !O.tree_cand || !O.tree_len)
        return fail(SENSE_ERR_INVALID_ARGUMENT,
                    "drafts, order, gamma, tree_tokens, tree_parent, tree_depth, tree_cand and "
                    "tree_len must be non-NULL");
    const int64_t nodes = (int64_t)(n_cand / n_groups) * max_len;
    if (O.mask && O.mask_ld < nodes)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "mask_ld = %lld < %lld nodes per group",
                    (long long)O.mask_ld, (long long)nodes);
    if (O.full_mask) {
        if (!dtype_ok(O.full_mask_dtype))
            return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown full_mask_dtype %d",
                        (int)O.full_mask_dtype);
        if (O.prefix_len < 0 || O.cache_len < 1)
            return fail(SENSE_ERR_INVALID_ARGUMENT, "prefix_len = %d and cache_len = %lld",
                        O.prefix_len, (long long)O.cache_len);
        if (!aligned(O.full_mask, (size_t)elem_size(O.full_mask_dtype)))
            return fail(SENSE_ERR_MISALIGNED, "full_mask not aligned to its element size");
    }
    sense::TrieOut T;
    T.order = O.order;
    T.gamma = O.gamma;
    T.tokens = O.tree_tokens;
    T.parent = O.tree_parent;
    T.depth = O.tree_depth;
    T.cand = O.tree_cand;
    T.tree_len = O.tree_len;
    T.sorted_drafts = O.sorted_drafts;
    T.sorted_len = O.sorted_len;
    T.mask = O.mask;
    T.mask_ld = O.mask_ld;
    T.full_mask = O.full_mask;
    T.full_dtype = O.full_mask_dtype;
    T.prefix_len = O.prefix_len;
    T.cache_len = O.full_mask ? O.cache_len : 0;
    hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    if ((e = timer_mark(SENSE_TIMER_TRIE, 0, st)) != hipSuccess) return hip_fail(e, "timer");
    e = sense::launch_trie(drafts, draft_len, n_cand, max_len, n_groups, T, st);
    if (e != hipSuccess) return hip_fail(e, "loose trie");
    if ((e = timer_mark(SENSE_TIMER_TRIE, 1, st)) != hipSuccess) return hip_fail(e, "timer");
    return ok();
}

SENSE_EXPORT sense_status_t sense_soft_gate_verify_tree_workspace_size(int32_t n_cand,
                                                                       int32_t max_len,
                                                                       int32_t vocab,
                                                                       int32_t n_groups,
                                                                       size_t* bytes) {
    if (!bytes) return fail(SENSE_ERR_INVALID_ARGUMENT, "bytes is NULL");
    sense_status_t s = check_verify_sizes(n_cand, max_len, vocab);
    if (s != SENSE_OK) return s;
    if (n_cand > 0 && (s = check_groups(n_cand, max_len, n_groups)) != SENSE_OK) return s;
    *bytes = sense::verify_tree_workspace_bytes(n_cand, max_len, vocab, n_groups);
    return ok();
}

SENSE_EXPORT sense_status_t sense_soft_gate_verify_tree(
    const void* logits, sense_dtype_t logits_dtype, int64_t row_stride,
    const int32_t* tree_tokens, const int32_t* tree_parent, const int32_t* tree_len,
    const int32_t* gamma, int32_t n_cand, int32_t max_len, int32_t vocab, int32_t n_groups,
    const sense_gate_params_t* params, int32_t* out_accept_len, int32_t* out_best,
    float* out_gate_score, uint8_t* out_masks, int32_t* out_rank, void* workspace,
    size_t workspace_bytes, void* stream) {
    sense_status_t s = check_verify_sizes(n_cand, max_len, vocab);
    if (s != SENSE_OK) return s;
    sense::GateParams gp;
    if ((s = check_gate_params(params, vocab, &gp)) != SENSE_OK) return s;
    if (!dtype_ok(logits_dtype))
        return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown logits dtype %d", (int)logits_dtype);
    if (row_stride < vocab)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "row_stride %lld < vocab %d", (long long)row_stride, vocab);
    if (n_cand == 0) return ok();
    if ((s = check_groups(n_cand, max_len, n_groups)) != SENSE_OK) return s;
    if (!logits || !tree_tokens || !tree_parent || !tree_len || !gamma || !out_accept_len ||
        !out_best)
        return fail(SENSE_ERR_INVALID_ARGUMENT,
                    "logits, tree_tokens, tree_parent, tree_len, gamma, out_accept_len and "
                    "out_best must be non-NULL");
    if (!aligned(logits, (size_t)elem_size(logits_dtype)))
        return fail(SENSE_ERR_MISALIGNED, "logits not aligned to their element size");
    const size_t need = sense::verify_tree_workspace_bytes(n_cand, max_len, vocab, n_groups);
    if (!workspace || workspace_bytes < need)
        return fail(SENSE_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 256)) return fail(SENSE_ERR_MISALIGNED, "workspace must be 256-byte aligned");
    hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    if ((e = timer_mark(SENSE_TIMER_VERIFY, 0, st)) != hipSuccess) return hip_fail(e, "timer");
    e = sense::launch_verify_tree(logits, logits_dtype, row_stride, tree_tokens, tree_parent,
                                  tree_len, gamma, n_cand, max_len, vocab, n_groups, gp,
                                  out_accept_len, out_best, out_gate_score, out_masks, out_rank,
                                  workspace, st);
    if (e != hipSuccess) return hip_fail(e, "soft-gated evaluation through the tree");
    if ((e = timer_mark(SENSE_TIMER_VERIFY, 1, st)) != hipSuccess) return hip_fail(e, "timer");
    return ok();
}

static sense_status_t check_projection(const sense_projection_t* p) {
    if (!p) return fail(SENSE_ERR_INVALID_ARGUMENT, "projection is NULL");
    if (!p->basis) return fail(SENSE_ERR_INVALID_ARGUMENT, "basis is NULL");
    if (p->d_in < 1 || p->d_in > sense::kMaxDim || p->d_in % 8 != 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "d_in = %d must be a multiple of 8 in [8, %d]",
                    p->d_in, sense::kMaxDim);
    if (p->d_out < 1 || p->d_out > sense::kMaxProjOut)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "d_out = %d outside [1, %d]", p->d_out,
                    sense::kMaxProjOut);
    if (!aligned(p->basis, 4) || (p->mean && !aligned(p->mean, 4)))
        return fail(SENSE_ERR_MISALIGNED, "basis and mean must be 4-byte aligned");
    return SENSE_OK;
}

SENSE_EXPORT sense_status_t sense_project_workspace_size(const sense_projection_t* proj,
                                                         sense_dtype_t x_dtype, int64_t n_rows,
                                                         size_t* bytes) {
    if (!bytes) return fail(SENSE_ERR_INVALID_ARGUMENT, "bytes is NULL");
    sense_status_t s = check_projection(proj);
    if (s != SENSE_OK) return s;
    if (!dtype_ok(x_dtype)) return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown x dtype %d", (int)x_dtype);
    if (n_rows < 0) return fail(SENSE_ERR_INVALID_ARGUMENT, "n_rows < 0");
    *bytes = sense::project_workspace_bytes(x_dtype, n_rows, proj->d_in, proj->d_out);
    return ok();
}

SENSE_EXPORT sense_status_t sense_project(const sense_projection_t* proj, const void* x,
                                          sense_dtype_t x_dtype, int64_t n_rows,
                                          int64_t x_stride, void* out, sense_dtype_t out_dtype,
                                          int64_t out_stride, void* workspace,
                                          size_t workspace_bytes, void* stream) {
    sense_status_t s = check_projection(proj);
    if (s != SENSE_OK) return s;
    if (!dtype_ok(x_dtype) || !dtype_ok(out_dtype))
        return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown dtype (x %d, out %d)", (int)x_dtype,
                    (int)out_dtype);
    if (n_rows < 0 || n_rows > 0x7FFFFFFFLL)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "n_rows = %lld outside [0, 2^31-1]",
                    (long long)n_rows);
    if (x_stride < proj->d_in || out_stride < proj->d_out)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "x_stride %lld < d_in or out_stride %lld < d_out",
                    (long long)x_stride, (long long)out_stride);
    if (n_rows == 0) return ok();
    if (!x || !out) return fail(SENSE_ERR_INVALID_ARGUMENT, "x and out must be non-NULL");
    if (!aligned(x, (size_t)elem_size(x_dtype)) || !aligned(out, (size_t)elem_size(out_dtype)))
        return fail(SENSE_ERR_MISALIGNED, "x or out not aligned to its element size");
    const size_t need = sense::project_workspace_bytes(x_dtype, n_rows, proj->d_in, proj->d_out);
    if (!workspace || workspace_bytes < need)
        return fail(SENSE_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 256)) return fail(SENSE_ERR_MISALIGNED, "workspace must be 256-byte aligned");
    hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    if ((e = timer_mark(SENSE_TIMER_PROJECT, 0, st)) != hipSuccess) return hip_fail(e, "timer");
    e = sense::launch_project(x, x_dtype, n_rows, proj->d_in, x_stride, proj->mean, proj->basis,
                              proj->d_out, proj->normalize, out, out_dtype, out_stride,
                              workspace, st);
    if (e != hipSuccess) return hip_fail(e, "projection");
    if ((e = timer_mark(SENSE_TIMER_PROJECT, 1, st)) != hipSuccess) return hip_fail(e, "timer");
    return ok();
}

// ------------------------------------------------------------ inverted file

static sense_status_t check_ivf_keys(const void* keys, sense_dtype_t key_dtype, int64_t n,
                                     int32_t d, int64_t key_stride) {
    if (key_dtype != SENSE_F16 && key_dtype != SENSE_BF16)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "key_dtype must be SENSE_F16 or SENSE_BF16");
    if (n < 1 || n > 0x7FFFFFFFLL)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "n = %lld outside [1, 2^31-1]", (long long)n);
    if (d < 8 || d > sense::kMaxIvfDim || d % 8 != 0)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "d = %d must be a multiple of 8 in [8, %d]", d,
                    sense::kMaxIvfDim);
    if (key_stride < d)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "key_stride %lld < d %d", (long long)key_stride, d);
    if (keys && (!aligned(keys, 16) || key_stride % 8 != 0))
        return fail(SENSE_ERR_MISALIGNED, "keys must be 16-byte aligned with key_stride %% 8 == 0");
    return SENSE_OK;
}

static sense_status_t check_pq(int32_t d, int32_t m, int32_t ksub) {
    if (m < 1 || d % m != 0 || d / m > sense::kMaxDsub)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "pq_m = %d must divide d = %d into <= %d dims", m,
                    d, sense::kMaxDsub);
    if (ksub < 1 || ksub > 256 || (int64_t)ksub * d > 16384)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "ksub = %d must be in [1, 256] with ksub * d <= 16384",
                    ksub);
    return SENSE_OK;
}

SENSE_EXPORT sense_status_t sense_ivf_assign(const void* keys, sense_dtype_t key_dtype, int64_t n,
                                             int32_t d, int64_t key_stride,
                                             const float* centroids, int32_t nlist,
                                             sense_metric_t metric, int32_t* out_list,
                                             void* stream) {
    sense_status_t s = check_ivf_keys(keys, key_dtype, n, d, key_stride);
    if (s != SENSE_OK) return s;
    if (!keys || !centroids || !out_list)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "keys, centroids and out_list must be non-NULL");
    if (nlist < 1 || nlist > sense::kMaxNlist)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "nlist = %d outside [1, %d]", nlist, sense::kMaxNlist);
    if (metric != SENSE_METRIC_IP && metric != SENSE_METRIC_COSINE)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown metric %d", (int)metric);
    if (!aligned(centroids, 4) || !aligned(out_list, 4))
        return fail(SENSE_ERR_MISALIGNED, "centroids and out_list must be 4-byte aligned");
    hipError_t e = sense::launch_ivf_assign(keys, key_dtype, n, d, key_stride, centroids, nlist,
                                            metric == SENSE_METRIC_COSINE, out_list,
                                            (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "ivf assign");
    return ok();
}

SENSE_EXPORT sense_status_t sense_pq_encode(const void* keys, sense_dtype_t key_dtype, int64_t n,
                                            int32_t d, int64_t key_stride,
                                            const float* centroids, int32_t nlist,
                                            const int32_t* list_ids, const float* codebooks,
                                            int32_t m, int32_t ksub, uint8_t* out_codes,
                                            void* stream) {
    sense_status_t s = check_ivf_keys(keys, key_dtype, n, d, key_stride);
    if (s != SENSE_OK) return s;
    if ((s = check_pq(d, m, ksub)) != SENSE_OK) return s;
    if (!keys || !centroids || !list_ids || !codebooks || !out_codes)
        return fail(SENSE_ERR_INVALID_ARGUMENT,
                    "keys, centroids, list_ids, codebooks and out_codes must be non-NULL");
    if (nlist < 1 || nlist > sense::kMaxNlist)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "nlist = %d outside [1, %d]", nlist, sense::kMaxNlist);
    if (!aligned(centroids, 4) || !aligned(codebooks, 4) || !aligned(list_ids, 4))
        return fail(SENSE_ERR_MISALIGNED, "centroids, codebooks and list_ids must be 4-byte aligned");
    hipError_t e = sense::launch_pq_encode(keys, key_dtype, n, d, key_stride, centroids, nlist,
                                           list_ids, codebooks, m, ksub, out_codes,
                                           (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "pq encode");
    return ok();
}

SENSE_EXPORT sense_status_t sense_build_ivf_index(const sense_ivf_desc_t* desc, void* stream,
                                                  sense_index_t** out) {
    if (!desc || !out) return fail(SENSE_ERR_INVALID_ARGUMENT, "desc and out must be non-NULL");
    *out = nullptr;
    const sense_ivf_desc_t& D = *desc;
    const bool pq = D.pq_codebooks != nullptr;
    sense_status_t s = check_ivf_keys(D.keys, D.key_dtype, D.n, D.d, D.key_stride);
    if (s != SENSE_OK) return s;
    if (pq && (s = check_pq(D.d, D.pq_m, D.pq_ksub)) != SENSE_OK) return s;
    if ((!pq && !D.keys) || (pq && !D.pq_codes) || !D.spans || !D.centroids || !D.list_ids)
        return fail(SENSE_ERR_INVALID_ARGUMENT,
                    "spans, centroids, list_ids and keys (IVF-Flat) or pq_codes (IVF-PQ) must be "
                    "non-NULL");
    if (D.nlist < 1 || D.nlist > sense::kMaxNlist)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "nlist = %d outside [1, %d]", D.nlist,
                    sense::kMaxNlist);
    if (D.max_span < 1 || D.max_span > sense::kMaxLen)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "max_span = %d outside [1, %d]", D.max_span,
                    sense::kMaxLen);
    if (D.metric != SENSE_METRIC_IP && D.metric != SENSE_METRIC_COSINE)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown metric %d", (int)D.metric);
    sense_index* ix = new (std::nothrow) sense_index();
    if (!ix) return fail(SENSE_ERR_OUT_OF_MEMORY, "host allocation failed");
    ix->key_dtype = D.key_dtype;
    ix->n = D.n;
    ix->d = D.d;
    ix->ld = D.d;
    ix->spans = D.spans;
    ix->max_span = D.max_span;
    ix->span_len = D.span_len;
    ix->span_stride = D.max_span;
    ix->metric = D.metric;
    ix->nlist = D.nlist;
    ix->pq_m = pq ? D.pq_m : 0;
    ix->pq_ksub = pq ? D.pq_ksub : 0;
    hipStream_t st = (hipStream_t)stream;
    const size_t n = (size_t)D.n, nl = (size_t)D.nlist;
    hipError_t e = hipSuccess;
    auto alloc = [&](void** p, size_t bytes) {
        if (e == hipSuccess) e = hipMalloc(p, bytes);
    };
    alloc((void**)&ix->centroids, nl * D.d * sizeof(float));
    alloc((void**)&ix->cen_inv, nl * sizeof(float));
    alloc((void**)&ix->counts, (nl + 2) * sizeof(int32_t));
    alloc((void**)&ix->cursor, nl * sizeof(int32_t));
    alloc((void**)&ix->offsets, (nl + 1) * sizeof(int64_t));
    alloc((void**)&ix->row_ids, n * sizeof(int32_t));
    if (pq) {
        alloc((void**)&ix->codes_sorted, n * D.pq_m);
        alloc((void**)&ix->codebooks, (size_t)D.pq_ksub * D.d * sizeof(float));
    } else {
        alloc(&ix->owned_keys, n * D.d * 2);
        if (D.metric == SENSE_METRIC_COSINE) alloc((void**)&ix->inv_norm, n * sizeof(float));
    }
    ix->cap_prefix = new (std::nothrow) int64_t[nl + 1];
    int32_t* host_counts = new (std::nothrow) int32_t[nl + 2];
    if (e != hipSuccess || !ix->cap_prefix || !host_counts) {
        delete[] host_counts;
        (void)sense_destroy_index(ix);
        return fail(SENSE_ERR_OUT_OF_MEMORY, "inverted-file index allocation failed");
    }
    ix->keys = ix->owned_keys;
    e = hipMemcpyAsync(ix->centroids, D.centroids, nl * D.d * sizeof(float),
                       hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess && pq)
        e = hipMemcpyAsync(ix->codebooks, D.pq_codebooks, (size_t)D.pq_ksub * D.d * sizeof(float),
                           hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess) e = sense::launch_f32_inv_norms(ix->centroids, D.nlist, D.d, ix->cen_inv, st);
    if (e == hipSuccess)
        e = sense::launch_ivf_layout(D.list_ids, D.n, D.nlist, D.keys, D.key_stride, D.d,
                                     D.pq_codes, ix->pq_m, ix->pq_ksub, ix->counts, ix->offsets,
                                     ix->cursor, ix->row_ids, pq ? nullptr : ix->owned_keys,
                                     ix->codes_sorted, st);
    if (e == hipSuccess && ix->inv_norm)
        e = sense::launch_key_norms(ix->owned_keys, D.key_dtype, D.n, D.d, D.d, ix->inv_norm,
                                    nullptr, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e == hipSuccess)
        e = hipMemcpy(host_counts, ix->counts, (nl + 2) * sizeof(int32_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) {
        delete[] host_counts;
        (void)sense_destroy_index(ix);
        return hip_fail(e, "inverted-file build");
    }
    if (host_counts[nl] != 0 || host_counts[nl + 1] != 0) {
        const int bad_l = host_counts[nl], bad_c = host_counts[nl + 1];
        delete[] host_counts;
        (void)sense_destroy_index(ix);
        return fail(SENSE_ERR_INVALID_ARGUMENT,
                    "%d list ids outside [0, %d) and %d codes >= pq_ksub", bad_l, D.nlist, bad_c);
    }
    // Sums of the p largest list sizes: the candidate slots nprobe lists can need.
    std::sort(host_counts, host_counts + nl, [](int32_t a, int32_t b) { return a > b; });
    ix->cap_prefix[0] = 0;
    for (size_t p = 0; p < nl; ++p) ix->cap_prefix[p + 1] = ix->cap_prefix[p] + host_counts[p];
    delete[] host_counts;
    *out = ix;
    return ok();
}

namespace {

struct IvfLayout {
    size_t q_off, coarse_off, ip_off, probe_off, pws_off, cnt_off, cand_off, total;
    int64_t cap;
};

IvfLayout ivf_layout(const sense_index* ix, int nq, int nprobe) {
    IvfLayout l;
    int64_t cap = ix->cap_prefix[nprobe];
    if (cap < 1) cap = 1;
    l.cap = cap;
    size_t at = 0;
    auto take = [&](size_t bytes) {
        const size_t o = at;
        at = round_up(at + bytes, 256);
        return o;
    };
    l.q_off = take((size_t)nq * ix->d * sizeof(float));
    l.coarse_off = take((size_t)nq * ix->nlist * sizeof(float));
    l.ip_off = take(ix->pq_m ? (size_t)nq * ix->nlist * sizeof(float) : 0);
    l.probe_off = take((size_t)nq * nprobe * sizeof(int64_t));
    l.pws_off = take(sense::topk_workspace_bytes(ix->nlist, nq, nprobe));
    l.cnt_off = take((size_t)nq * sizeof(int32_t));
    l.cand_off = take((size_t)nq * cap * sizeof(uint64_t));
    l.total = at;
    return l;
}

}  // namespace

static sense_status_t check_ivf_search(const sense_index_t* ix, int32_t nq, int32_t k,
                                       int32_t nprobe) {
    if (!ix) return fail(SENSE_ERR_INVALID_ARGUMENT, "index is NULL");
    if (ix->nlist < 1) return fail(SENSE_ERR_INVALID_ARGUMENT, "index is not an inverted file");
    if (nq < 1) return fail(SENSE_ERR_INVALID_ARGUMENT, "n_queries = %d < 1", nq);
    if (k < 1) return fail(SENSE_ERR_INVALID_ARGUMENT, "k = %d < 1", k);
    if (k > sense::kMaxK) return fail(SENSE_ERR_UNSUPPORTED, "k = %d > %d", k, sense::kMaxK);
    if (nprobe < 1 || nprobe > ix->nlist)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "nprobe = %d outside [1, %d]", nprobe, ix->nlist);
    if (nprobe > sense::kMaxK) return fail(SENSE_ERR_UNSUPPORTED, "nprobe = %d > %d", nprobe, sense::kMaxK);
    return SENSE_OK;
}

SENSE_EXPORT sense_status_t sense_ivf_search_workspace_size(const sense_index_t* ix, int32_t nq,
                                                            int32_t k, int32_t nprobe,
                                                            size_t* bytes) {
    if (!bytes) return fail(SENSE_ERR_INVALID_ARGUMENT, "bytes is NULL");
    const sense_status_t s = check_ivf_search(ix, nq, k, nprobe);
    if (s != SENSE_OK) return s;
    *bytes = ivf_layout(ix, nq, nprobe).total;
    return ok();
}

SENSE_EXPORT sense_status_t sense_ivf_search(const sense_index_t* ix, const void* queries,
                                             sense_dtype_t q_dtype, int32_t nq, int32_t k,
                                             int32_t nprobe, int64_t* out_ids, float* out_scores,
                                             int32_t* out_drafts, int32_t* out_draft_len,
                                             int64_t* out_probe, void* workspace,
                                             size_t workspace_bytes, void* stream) {
    sense_status_t s = check_ivf_search(ix, nq, k, nprobe);
    if (s != SENSE_OK) return s;
    if (!queries || !out_ids)
        return fail(SENSE_ERR_INVALID_ARGUMENT, "queries and out_ids must be non-NULL");
    if (!dtype_ok(q_dtype)) return fail(SENSE_ERR_INVALID_ARGUMENT, "unknown q_dtype %d", (int)q_dtype);
    if (!aligned(queries, q_dtype == SENSE_F32 ? 16 : 2))
        return fail(SENSE_ERR_MISALIGNED, "fp32 queries must be 16-byte aligned");
    const IvfLayout L = ivf_layout(ix, nq, nprobe);
    if (!workspace || workspace_bytes < L.total)
        return fail(SENSE_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", L.total,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 256)) return fail(SENSE_ERR_MISALIGNED, "workspace must be 256-byte aligned");
    hipStream_t st = (hipStream_t)stream;
    char* ws = (char*)workspace;
    hipError_t e;
    const float* qptr = (const float*)queries;
    if (q_dtype != SENSE_F32) {
        if ((e = sense::launch_query_to_f32(queries, q_dtype, nq, ix->d, (float*)(ws + L.q_off),
                                            st)) != hipSuccess)
            return hip_fail(e, "query conversion");
        qptr = (const float*)(ws + L.q_off);
    }
    sense::IvfSearch S{};
    S.queries = qptr;
    S.d = ix->d;
    S.nq = nq;
    S.centroids = ix->centroids;
    S.cen_inv = ix->cen_inv;
    S.nlist = ix->nlist;
    S.cosine = ix->metric == SENSE_METRIC_COSINE;
    S.coarse = (float*)(ws + L.coarse_off);
    S.coarse_ip = ix->pq_m ? (float*)(ws + L.ip_off) : nullptr;
    S.probe = out_probe ? out_probe : (int64_t*)(ws + L.probe_off);
    S.probe_ws = ws + L.pws_off;
    S.nprobe = nprobe;
    S.offsets = ix->offsets;
    S.count = (int32_t*)(ws + L.cnt_off);
    S.cap = L.cap;
    S.cand = (uint64_t*)(ws + L.cand_off);
    S.codes_sorted = ix->codes_sorted;
    S.m = ix->pq_m;
    S.ksub = ix->pq_ksub;
    S.codebooks = ix->codebooks;
    S.keys_sorted = ix->owned_keys;
    S.key_dtype = ix->key_dtype;
    S.inv_norm = ix->inv_norm;
    S.row_ids = ix->row_ids;
    S.k = k;
    S.spans = ix->spans;
    S.span_len = ix->span_len;
    S.max_span = ix->max_span;
    S.span_stride = ix->span_stride;
    S.out_ids = out_ids;
    S.out_scores = out_scores;
    S.out_drafts = out_drafts;
    S.out_draft_len = out_draft_len;
    if ((e = timer_mark(SENSE_TIMER_IVF, 0, st)) != hipSuccess) return hip_fail(e, "timer");
    if ((e = sense::launch_ivf_search(S, st)) != hipSuccess) return hip_fail(e, "ivf search");
    if ((e = timer_mark(SENSE_TIMER_IVF, 1, st)) != hipSuccess) return hip_fail(e, "timer");
    return ok();
}
