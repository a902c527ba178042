// Candidate selection around the retrieval (Sec. 3.2 Eq. 8; Alg. 2's hybrid
// retrieval, composite score, Top-N and anchor override).
//
// Per query, the pool D_all is the static hits followed by the dynamic-cache
// hits.  Each member gets the composite score
//     S_i = alpha * I(first token == anchor) + beta * s_i,
// with s_i the static similarity or the dynamic similarity plus the boost
// delta, taken in binary32 as one fused multiply-add (the delta addition
// rounds separately).  A draft of length <= 0 has no first token.  The top_n
// members by (S desc, position asc; NaN last) become the draft pool, and the
// override writes the anchor into the first token of the pool's first and
// last drafts (a draft of length 0 then has length 1), so both start with the
// model's greedy token.
//
// One block per query.  The pool is at most kMaxPool members, so the whole
// ranking is one bitonic sort of packed 64-bit keys (score bits, complemented
// position) in LDS; the gather copies the chosen rows with one thread per
// output token.
#include "internal.h"

namespace sense {
namespace {

constexpr int kSelThreads = 256;

__global__ __launch_bounds__(kSelThreads) void select_candidates_kernel(
    const float* __restrict__ scores_s, const int32_t* __restrict__ drafts_s,
    const int32_t* __restrict__ len_s, int n_s, const float* __restrict__ scores_d,
    const int32_t* __restrict__ drafts_d, const int32_t* __restrict__ len_d, int n_d,
    const int32_t* __restrict__ anchors, int max_len, int top_n, SelectParams sp,
    int32_t* __restrict__ out_drafts, int32_t* __restrict__ out_len,
    int32_t* __restrict__ out_source, float* __restrict__ out_score) {
    __shared__ uint64_t s_key[kMaxPool];
    const int q = blockIdx.x;
    const int n_all = n_s + n_d;
    int p = 1;
    while (p < n_all) p <<= 1;
    const int32_t anchor = anchors[q];

    for (int i = threadIdx.x; i < p; i += kSelThreads) {
        uint64_t key = 0;  // padding: below every member
        if (i < n_all) {
            const bool dyn = i >= n_s;
            const int r = dyn ? i - n_s : i;
            const int64_t row = (int64_t)q * (dyn ? n_d : n_s) + r;
            const int32_t* lens = dyn ? len_d : len_s;
            const int len = lens ? lens[row] : max_len;
            const int32_t first = (dyn ? drafts_d : drafts_s)[row * max_len];
            const bool match = len > 0 && first == anchor;
            const float s = dyn ? scores_d[row] + sp.delta : scores_s[row];
            const float S = __builtin_fmaf(sp.beta, s, match ? sp.alpha : 0.0f);
            key = pack_key(S, (uint32_t)i);
        }
        s_key[i] = key;
    }
    __syncthreads();
    bitonic_desc<kSelThreads>(s_key, p);

    for (int t = threadIdx.x; t < top_n * max_len; t += kSelThreads) {
        const int r = t / max_len, j = t - r * max_len;
        const uint64_t key = s_key[r];
        const int i = (int)key_row(key);
        const bool dyn = i >= n_s;
        const int src = dyn ? i - n_s : i;
        const int64_t row = (int64_t)q * (dyn ? n_d : n_s) + src;
        const int32_t* lens = dyn ? len_d : len_s;
        int len = lens ? lens[row] : max_len;
        len = len < 0 ? 0 : (len > max_len ? max_len : len);
        int32_t v = j < len ? (dyn ? drafts_d : drafts_s)[row * max_len + j] : -1;
        const bool pinned = sp.anchor_override && (r == 0 || r == top_n - 1);
        if (pinned && j == 0) v = anchor;
        const int64_t o = (int64_t)q * top_n + r;
        out_drafts[o * max_len + j] = v;
        if (j == 0) {
            out_len[o] = (pinned && len < 1) ? 1 : len;
            if (out_source) out_source[o] = i;
            if (out_score) out_score[o] = key_score((uint32_t)(key >> 32));
        }
    }
}

}  // namespace

hipError_t launch_select_candidates(const float* scores_s, const int32_t* drafts_s,
                                    const int32_t* len_s, int n_s, const float* scores_d,
                                    const int32_t* drafts_d, const int32_t* len_d, int n_d,
                                    const int32_t* anchors, int n_queries, int max_len,
                                    int top_n, const SelectParams& sp, int32_t* out_drafts,
                                    int32_t* out_len, int32_t* out_source, float* out_score,
                                    hipStream_t stream) {
    hipLaunchKernelGGL(select_candidates_kernel, dim3(n_queries), dim3(kSelThreads), 0, stream,
                       scores_s, drafts_s, len_s, n_s, scores_d, drafts_d, len_d, n_d, anchors,
                       max_len, top_n, sp, out_drafts, out_len, out_source, out_score);
    return hipGetLastError();
}

}  // namespace sense
