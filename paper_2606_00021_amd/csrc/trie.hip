// Loose trie of a candidate pool (Sec. 3.2 Eq. 9 and the tree mask after
// it; Alg. 2's LexSort; Alg. 3; the static-KV tree mask of the appendix).
//
// trie_build: one block per candidate group (at most 1024 drafts and 4096
//   draft tokens, all held in LDS):
//     1. LexSort of the draft indices by their token sequences (a proper
//        prefix first, identical drafts by index): groups of up to 256
//        drafts place each draft at the count of drafts before it (all
//        pairs in one round), larger ones use a bitonic network;
//     2. prefix detection: sorted draft r position j repeats draft r-1 when
//        both exist and every token up to j is equal (the running product
//        along the row);
//     3. tree extraction and index map: an exclusive block scan of the
//        "new token" flags in row-major order numbers the tree tokens; a
//        shared position takes the latest number above it in its column
//        (a max-scan down the rows: across the lanes of one wave per column
//        for up to 64 drafts, else log2 N doubling steps);
//     4. outputs: the permutation, Gamma, and per tree token its id, parent,
//        depth and the sorted draft that creates it (the inverse map).
//   Numbering in row-major order of lexicographically sorted drafts visits
//   the tree in preorder.
// trie_mask: one block per (tree token, group): row u of the ancestor mask
//   (v is on u's path when depth(v) <= depth(u) and Gamma of u's draft at
//   depth(v) is v) and, if asked, row u of the static-KV mask, additive
//   0 / -inf over the cache.
#include "internal.h"

namespace sense {
namespace {

constexpr int kTrieThreads = 1024;
constexpr int kTriePer = kMaxNodes / kTrieThreads;   // elements per thread (4)
constexpr int kRankSortMax = 256;   // groups up to this size are ranked by counting

// Draft a sorts before draft b: lexicographic on the sequences, then index.
// Indices >= n are padding and sort after every draft.
__device__ inline bool lex_less(int a, int b, int n, int m, const int32_t* s_d,
                                const int32_t* s_len) {
    if (a >= n) return false;
    if (b >= n) return true;
    const int la = s_len[a], lb = s_len[b];
    const int l = la < lb ? la : lb;
    for (int j = 0; j < l; ++j) {
        const int32_t ta = s_d[a * m + j], tb = s_d[b * m + j];
        if (ta != tb) return ta < tb;
    }
    if (la != lb) return la < lb;
    return a < b;
}

__global__ __launch_bounds__(kTrieThreads) void trie_build_kernel(
    const int32_t* __restrict__ drafts, const int32_t* __restrict__ draft_len, int gs, int m,
    TrieOut out) {
    __shared__ int32_t s_d[kMaxNodes];        // the group's drafts, original order
    __shared__ int32_t s_flag[kMaxNodes];     // new-token flags, sorted row-major
    __shared__ int32_t s_idx[kMaxNodes];      // tree ids, then Gamma
    __shared__ int32_t s_len[kMaxGroup];
    __shared__ int32_t s_perm[kMaxGroup];
    __shared__ int32_t s_wave[kTrieThreads / 64];
    const int g = blockIdx.x;
    const int tid = threadIdx.x;
    const int nodes = gs * m;
    const int64_t cand0 = (int64_t)g * gs;

    for (int t = tid; t < nodes; t += kTrieThreads) s_d[t] = drafts[cand0 * m + t];
    int p = 1;
    while (p < gs) p <<= 1;
    for (int r = tid; r < p; r += kTrieThreads) {
        if (r < gs) {
            int l = draft_len ? draft_len[cand0 + r] : m;
            s_len[r] = l < 0 ? 0 : (l > m ? m : l);
        }
        s_perm[r] = r;
    }
    __syncthreads();

    // 1. LexSort.  Small groups: every draft's place is the number of drafts
    //    before it (all pairs compared at once, one round).  Larger groups:
    //    an ascending bitonic network over p entries.
    if (gs <= kRankSortMax) {
        for (int r = tid; r < gs; r += kTrieThreads) s_idx[r] = 0;
        __syncthreads();
        const int pairs = gs * gs;
        const int per = (pairs + kTrieThreads - 1) / kTrieThreads;
        int a_cur = -1, cnt = 0;
        for (int t = tid * per; t < pairs && t < (tid + 1) * per; ++t) {
            const int a = t / gs, b = t - a * gs;
            if (a != a_cur) {
                if (cnt) atomicAdd(&s_idx[a_cur], cnt);
                a_cur = a;
                cnt = 0;
            }
            cnt += (b != a && lex_less(b, a, gs, m, s_d, s_len)) ? 1 : 0;
        }
        if (cnt) atomicAdd(&s_idx[a_cur], cnt);
        __syncthreads();
        for (int r = tid; r < gs; r += kTrieThreads) s_perm[s_idx[r]] = r;
        __syncthreads();
        p = 1;                           // the network below is skipped
    }
    for (int size = 2; size <= p; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = tid; i < (p >> 1); i += kTrieThreads) {
                const int pos = 2 * i - (i & (stride - 1));
                const int partner = pos + stride;
                const bool asc = (pos & size) == 0;
                const int a = s_perm[pos], b = s_perm[partner];
                const bool a_after_b = lex_less(b, a, gs, m, s_d, s_len);
                if (a_after_b == asc) {
                    s_perm[pos] = b;
                    s_perm[partner] = a;
                }
            }
            __syncthreads();
        }
    }

    // 2. Prefix detection, one thread per sorted draft.
    for (int r = tid; r < gs; r += kTrieThreads) {
        const int a = s_perm[r];
        const int b = r > 0 ? s_perm[r - 1] : -1;
        const int la = s_len[a], lb = b >= 0 ? s_len[b] : 0;
        bool run = true;
        for (int j = 0; j < m; ++j) {
            const bool exists = j < la;
            run = run && exists && j < lb && s_d[a * m + j] == s_d[b * m + j];
            s_flag[r * m + j] = (exists && !run) ? 1 : 0;
        }
    }
    __syncthreads();

    // 3a. Exclusive scan of the flags: thread tid owns elements
    //     [kTriePer * tid, kTriePer * tid + kTriePer).
    int f[kTriePer];
    int local = 0;
#pragma unroll
    for (int e = 0; e < kTriePer; ++e) {
        const int t = kTriePer * tid + e;
        f[e] = t < nodes ? s_flag[t] : 0;
        local += f[e];
    }
    const int lane = tid & 63, wv = tid >> 6;
    int incl = local;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off, 64);
        if (lane >= off) incl += y;
    }
    if (lane == 63) s_wave[wv] = incl;
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wv; ++w) before += s_wave[w];
    int total = 0;
    for (int w = 0; w < kTrieThreads / 64; ++w) total += s_wave[w];
    int run_id = before + incl - local;
#pragma unroll
    for (int e = 0; e < kTriePer; ++e) {
        const int t = kTriePer * tid + e;
        if (t < nodes) s_idx[t] = f[e] ? run_id : -1;
        run_id += f[e];
    }
    __syncthreads();
    const int L = total;

    // 3b. Max-scan down the rows of every column.  Up to 64 rows: one wave
    //     per column, lane r holding row r, an inclusive max-scan across the
    //     lanes (columns are independent).  More rows: Hillis-Steele doubling
    //     over the block.
    if (gs <= 64) {
        for (int j = wv; j < m; j += kTrieThreads / 64) {
            const int t = lane * m + j;
            int v = lane < gs ? s_idx[t] : -1;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int y = __shfl_up(v, off, 64);
                if (lane >= off) v = v > y ? v : y;
            }
            if (lane < gs) s_idx[t] = v;
        }
        __syncthreads();
    }
    for (int s = 1; s < (gs <= 64 ? 1 : gs); s <<= 1) {
        int v[kTriePer];
#pragma unroll
        for (int e = 0; e < kTriePer; ++e) {
            const int t = kTriePer * tid + e;
            v[e] = -1;
            if (t < nodes) {
                const int up = t - s * m;
                v[e] = s_idx[t];
                if (up >= 0) v[e] = v[e] > s_idx[up] ? v[e] : s_idx[up];
            }
        }
        __syncthreads();
#pragma unroll
        for (int e = 0; e < kTriePer; ++e) {
            const int t = kTriePer * tid + e;
            if (t < nodes) s_idx[t] = v[e];
        }
        __syncthreads();
    }

    // 4. Outputs.
    const int64_t node0 = (int64_t)g * nodes;
    for (int t = tid; t < nodes; t += kTrieThreads) {
        const int r = t / m, j = t - r * m;
        const int a = s_perm[r];
        const bool exists = j < s_len[a];
        const int gam = exists ? s_idx[t] : -1;
        out.gamma[(cand0 + r) * m + j] = gam;
        if (out.sorted_drafts) out.sorted_drafts[(cand0 + r) * m + j] = exists ? s_d[a * m + j] : -1;
        if (s_flag[t]) {
            const int64_t u = node0 + gam;
            out.tokens[u] = s_d[a * m + j];
            out.parent[u] = j > 0 ? s_idx[t - 1] : -1;
            out.depth[u] = j;
            out.cand[u] = r;
        }
    }
    for (int u = L + tid; u < nodes; u += kTrieThreads) {
        out.tokens[node0 + u] = -1;
        out.parent[node0 + u] = -1;
        out.depth[node0 + u] = -1;
        out.cand[node0 + u] = -1;
    }
    for (int r = tid; r < gs; r += kTrieThreads) {
        out.order[cand0 + r] = s_perm[r];
        if (out.sorted_len) out.sorted_len[cand0 + r] = s_len[s_perm[r]];
    }
    if (tid == 0) out.tree_len[g] = L;
}

constexpr int kMaskThreads = 256;

__device__ inline void store_full(void* base, int dt, int64_t i, bool visible) {
    if (dt == DT_F32) {
        ((float*)base)[i] = visible ? 0.0f : -__builtin_inff();
    } else {
        // -inf: binary16 0xFC00, bfloat16 0xFF80; +0 in both is 0x0000.
        const uint16_t ninf = dt == DT_F16 ? (uint16_t)0xFC00u : (uint16_t)0xFF80u;
        ((uint16_t*)base)[i] = visible ? (uint16_t)0 : ninf;
    }
}

__global__ __launch_bounds__(kMaskThreads) void trie_mask_kernel(int gs, int m, TrieOut out) {
    const int u = blockIdx.x, g = blockIdx.y;
    const int L = out.tree_len[g];
    if (u >= L) return;                              // uniform over the block
    const int nodes = gs * m;
    const int64_t node0 = (int64_t)g * nodes;
    const int r = out.cand[node0 + u];
    const int du = out.depth[node0 + u];
    const int32_t* path = out.gamma + ((int64_t)g * gs + r) * m;
    auto on_path = [&](int v) {
        const int dv = out.depth[node0 + v];
        return dv >= 0 && dv <= du && path[dv] == v;
    };
    if (out.mask) {
        uint8_t* row = out.mask + (node0 + u) * out.mask_ld;
        for (int v = threadIdx.x; v < L; v += kMaskThreads) row[v] = on_path(v) ? 1 : 0;
    }
    if (out.full_mask) {
        const int64_t row0 = (node0 + u) * out.cache_len;
        for (int64_t c = threadIdx.x; c < out.cache_len; c += kMaskThreads) {
            bool vis;
            if (c < out.prefix_len) vis = true;
            else if (c < (int64_t)out.prefix_len + L) vis = on_path((int)(c - out.prefix_len));
            else vis = false;
            store_full(out.full_mask, out.full_dtype, row0 + c, vis);
        }
    }
}

}  // namespace

hipError_t launch_trie(const int32_t* drafts, const int32_t* draft_len, int n_cand, int max_len,
                       int n_groups, const TrieOut& out, hipStream_t stream) {
    const int gs = n_cand / n_groups;
    hipLaunchKernelGGL(trie_build_kernel, dim3((unsigned)n_groups), dim3(kTrieThreads), 0,
                       stream, drafts, draft_len, gs, max_len, out);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || (!out.mask && !out.full_mask)) return e;
    hipLaunchKernelGGL(trie_mask_kernel, dim3((unsigned)(gs * max_len), (unsigned)n_groups),
                       dim3(kMaskThreads), 0, stream, gs, max_len, out);
    return hipGetLastError();
}

}  // namespace sense
