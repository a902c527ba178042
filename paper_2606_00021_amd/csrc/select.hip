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
// One block per query.  The pool is at most kMaxPool members, ranked as
// packed 64-bit keys (score bits, complemented position) in LDS: up to 256
// members by rank (each counts the members above it), more by a bitonic
// sort; the gather copies the chosen rows, one thread per output token.
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

    // Member i's row: static hits first, then the dynamic ones.  Loads are
    // unconditional (a missing length table reads the draft's first token,
    // a valid address, and is then ignored), so each thread's loads are in
    // flight together.
    auto member = [&](int i, int64_t& row, const int32_t*& dsrc, int& len) {
        const bool dyn = i >= n_s;
        row = (int64_t)q * (dyn ? n_d : n_s) + (dyn ? i - n_s : i);
        dsrc = (dyn ? drafts_d : drafts_s) + row * max_len;
        const int32_t* lens = dyn ? len_d : len_s;
        const int lraw = *(lens ? lens + row : dsrc);
        len = lens ? lraw : max_len;
    };
    for (int i = threadIdx.x; i < p; i += kSelThreads) {
        const int ic = i < n_all ? i : n_all - 1;
        int64_t row;
        const int32_t* dsrc;
        int len;
        member(ic, row, dsrc, len);
        const bool dyn = ic >= n_s;
        const int32_t first = dsrc[0];
        const float sv = (dyn ? scores_d : scores_s)[row];
        const bool match = len > 0 && first == anchor;
        const float sc = dyn ? sv + sp.delta : sv;
        const float S = __builtin_fmaf(sp.beta, sc, match ? sp.alpha : 0.0f);
        s_key[i] = i < n_all ? pack_key(S, (uint32_t)i) : 0;   // padding: below every member
    }
    __syncthreads();
    if (n_all <= kSelThreads) {
        // Rank sort: each member counts the members above it (LDS broadcast
        // reads; keys are unique, so the ranks are a permutation).
        uint64_t mine = 0;
        int rank = 0;
        if (threadIdx.x < n_all) {
            mine = s_key[threadIdx.x];
            for (int j = 0; j < n_all; ++j) rank += s_key[j] > mine ? 1 : 0;
        }
        __syncthreads();
        if (threadIdx.x < n_all) s_key[rank] = mine;
        __syncthreads();
    } else {
        bitonic_desc<kSelThreads>(s_key, p);
    }

    // Gather: kOut outputs per thread and round, every load requested before
    // any store (rank r < top_n <= n_all holds a member).
    constexpr int kOut = 4;
    const int total = top_n * max_len;
    for (int t0 = 0; t0 < total; t0 += kOut * kSelThreads) {
        int32_t dv[kOut], lv[kOut], iv[kOut];
#pragma unroll
        for (int u = 0; u < kOut; ++u) {
            const int t = t0 + threadIdx.x + u * kSelThreads;
            const int tc = t < total ? t : total - 1;
            const int r = tc / max_len, j = tc - r * max_len;
            const int i = (int)key_row(s_key[r]);
            int64_t row;
            const int32_t* dsrc;
            member(i, row, dsrc, lv[u]);
            dv[u] = dsrc[j];
            iv[u] = i;
        }
#pragma unroll
        for (int u = 0; u < kOut; ++u) {
            const int t = t0 + threadIdx.x + u * kSelThreads;
            if (t >= total) continue;
            const int r = t / max_len, j = t - r * max_len;
            int len = lv[u];
            len = len < 0 ? 0 : (len > max_len ? max_len : len);
            int32_t v = j < len ? dv[u] : -1;
            const bool pinned = sp.anchor_override && (r == 0 || r == top_n - 1);
            if (pinned && j == 0) v = anchor;
            const int64_t o = (int64_t)q * top_n + r;
            out_drafts[o * max_len + j] = v;
            if (j == 0) {
                out_len[o] = (pinned && len < 1) ? 1 : len;
                if (out_source) out_source[o] = iv[u];
                if (out_score) out_score[o] = key_score((uint32_t)(s_key[r] >> 32));
            }
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
