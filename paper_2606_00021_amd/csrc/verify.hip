// Soft-gated evaluation (Sec. 3.3 Eqs. 12-18; Alg. 4) of a candidate draft
// batch against the target's aligned logits.
//
// The cost is one read of the logits of every live (candidate, position)
// row; everything else is per-row scalars.  Two kernels:
//
// verify_rows: one block of 256 threads per (row, vocabulary slice).  A
//   slice is what the block holds in registers: every thread issues all of
//   its eight 16-byte loads at once (no dependent chain; small blocks keep
//   the register count low, so many blocks share a compute unit and one's
//   arithmetic hides another's loads), then
//     phase 1: m = max of the slice (wave max, then the four waves);
//     phase 2: with t = (x - m) log2 e,
//       S   = sum 2^t                 (= sum e^(x-m)),
//       T2  = sum 2^t * t             (= log2 e * sum e^(x-m)(x-m)),
//       cnt = #{v : x_v > x_d} + #{v < d : x_v = x_d},  x_d the draft token's
//             logit, counted as x_v >= x_d left of d and x_v >= next(x_d)
//             from d on (one compare per element; in a full slice a wave
//             ballot per element, counted on the scalar unit).
//   and stores one 16-byte partial (m, S, T2, cnt) per (row, slice).  With
//   p = softmax(x), E = -sum p ln p = ln S - ln2 * T2 / S.  The draft token
//   is the first argmax exactly when cnt = 0 and is in the top-k set exactly
//   when cnt < k, so neither an argmax nor a sort of the vocabulary is needed.
//   Sums are formed in a fixed order (DPP butterflies, then the waves in
//   order), so results are deterministic.
//
// verify_finalize: one block per candidate group.  Phase 1 gives every
//   (candidate, position) row its own thread, which merges the row's slices
//   in slice order and forms the exact-match / entropy / top-k bits; phase 2
//   gives every row a thread again, which counts its window's mismatches
//   with one popcount over the candidate's 64-bit exact-match mask and forms
//   its gate bit; phase 3 gives every candidate a thread that takes the
//   leading run of its gate mask; the block then picks the group's first
//   longest candidate.
#include "internal.h"

namespace sense {
namespace {

constexpr int kRowThreads = kVerifyRowThreads;
constexpr int kRowWaves = kRowThreads / 64;
constexpr int kNV = 8;             // 16-byte vectors per thread per slice
constexpr int kScalarPer = 32;     // elements per thread per slice, unaligned rows
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct Partial {
    float m;
    float s;
    float t2;
    int cnt;
};

struct Stats {
    float m, s, t2;
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Merge of two (m, S, T2) states of disjoint element sets.
__device__ __forceinline__ Stats merge(const Stats& a, const Stats& b) {
    if (a.m == -__builtin_inff()) return b;
    if (b.m == -__builtin_inff()) return a;
    const float mm = a.m > b.m ? a.m : b.m;
    const float da = (a.m - mm) * kLog2e, db = (b.m - mm) * kLog2e;
    const float fa = fast_exp2(da), fb = fast_exp2(db);
    Stats r;
    r.m = mm;
    r.s = fa * a.s + fb * b.s;
    r.t2 = fa * __builtin_fmaf(da, a.s, a.t2) + fb * __builtin_fmaf(db, b.s, b.t2);
    return r;
}

template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
    return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __builtin_bit_cast(float, dpp_i<CTRL>(__builtin_bit_cast(int, x)));
}
__device__ __forceinline__ float lane_f(float x, int lane) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), lane));
}

// Wave-uniform sum / max over 64 lanes in a fixed order.
__device__ __forceinline__ float wave_sum_f(float x) {
    x += dpp_f<0xB1>(x);
    x += dpp_f<0x4E>(x);
    x += dpp_f<0x141>(x);
    x += dpp_f<0x140>(x);
    return (lane_f(x, 0) + lane_f(x, 16)) + (lane_f(x, 32) + lane_f(x, 48));
}
__device__ __forceinline__ int wave_sum_i(int x) {
    x += dpp_i<0xB1>(x);
    x += dpp_i<0x4E>(x);
    x += dpp_i<0x141>(x);
    x += dpp_i<0x140>(x);
    return (__builtin_amdgcn_readlane(x, 0) + __builtin_amdgcn_readlane(x, 16)) +
           (__builtin_amdgcn_readlane(x, 32) + __builtin_amdgcn_readlane(x, 48));
}
__device__ __forceinline__ float wave_max_f(float x) {
    x = __builtin_fmaxf(x, dpp_f<0xB1>(x));
    x = __builtin_fmaxf(x, dpp_f<0x4E>(x));
    x = __builtin_fmaxf(x, dpp_f<0x141>(x));
    x = __builtin_fmaxf(x, dpp_f<0x140>(x));
    return __builtin_fmaxf(__builtin_fmaxf(lane_f(x, 0), lane_f(x, 16)),
                           __builtin_fmaxf(lane_f(x, 32), lane_f(x, 48)));
}

template <int LT>
__device__ __forceinline__ float load_one(const char* base, int64_t i) {
    if constexpr (LT == DT_F32) {
        return ((const float*)base)[i];
    } else if constexpr (LT == DT_BF16) {
        return __builtin_bit_cast(float, (uint32_t)((const uint16_t*)base)[i] << 16);
    } else {
        return (float)__builtin_bit_cast(_Float16, ((const uint16_t*)base)[i]);
    }
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int LT>
__device__ __forceinline__ void unpack(const u32x4& w, float (&x)[LT == DT_F32 ? 4 : 8]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        // Copy the lane out first: a bit_cast applied directly to an element
        // of an ext_vector_type is mis-compiled by this hipcc (it reads the
        // wrong element).
        const uint32_t u = w[i];
        if constexpr (LT == DT_F32) {
            x[i] = __builtin_bit_cast(float, u);
        } else if constexpr (LT == DT_BF16) {
            x[2 * i] = __builtin_bit_cast(float, u << 16);
            x[2 * i + 1] = __builtin_bit_cast(float, u & 0xFFFF0000u);
        } else {
            x[2 * i] = (float)__builtin_bit_cast(_Float16, (uint16_t)(u & 0xFFFFu));
            x[2 * i + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(u >> 16));
        }
    }
}

// Threshold of "x > x_d" as "x >= next_up(x_d)": the smallest float above a
// finite or -inf x.  Nothing lies above +inf, so there it is NaN, which no
// comparison reaches (elements from d on that equal +inf rank below d, as in
// the stable order); NaN maps to itself.
__device__ __forceinline__ float next_up(float x) {
    if (x != x) return x;
    if (x == __builtin_inff()) return __builtin_nanf("");
    if (x == 0.0f) return __builtin_bit_cast(float, 1u);
    const uint32_t u = __builtin_bit_cast(uint32_t, x);
    return __builtin_bit_cast(float, x > 0.0f ? u + 1u : u - 1u);
}

// Maximum and fixed-order pairwise sums over the block's per-wave values.
__device__ __forceinline__ float waves_max(const float* s) {
    float m = s[0];
#pragma unroll
    for (int w = 1; w < kRowWaves; ++w) m = __builtin_fmaxf(m, s[w]);
    return m;
}
template <int N, typename T, typename Get>
__device__ __forceinline__ T pair_sum(Get get, int off) {
    if constexpr (N == 1) {
        return get(off);
    } else {
        return pair_sum<N / 2, T>(get, off) + pair_sum<N / 2, T>(get, off + N / 2);
    }
}

struct Acc {
    float s = 0.0f, t2 = 0.0f;
    int cnt = 0;        // per lane
    uint32_t wcnt = 0;  // per wave (already summed over its lanes)
};

// One element of phase 2.  The clamp keeps a -inf logit at weight 0 and
// contribution 0 (instead of 0 * -inf).
__device__ __forceinline__ void absorb_sum(Acc& a, float x, float nm) {
    const float t = __builtin_fmaxf(__builtin_fmaf(x, kLog2e, nm), -256.0f);
    const float e = fast_exp2(t);
    a.s += e;
    a.t2 = __builtin_fmaf(e, t, a.t2);
}
__device__ __forceinline__ void absorb(Acc& a, float x, float nm, float thr) {
    absorb_sum(a, x, nm);
    a.cnt += (x >= thr) ? 1 : 0;
}

// One block per (item, vocabulary slice).  Dense: item = candidate * max_len
// + position, its own logits row, token drafts[item].  TREE: item = group *
// nodes + u, token tree_tokens[item]; it is judged when u < tree_len[group]
// and its parent is a node of the group (or none), and its logits row is
// 1 + parent within the group's 1 + nodes rows.
template <int LT, bool VEC, bool TREE>
__global__ __launch_bounds__(kRowThreads) void verify_rows_kernel(
    const void* __restrict__ logits, int64_t row_stride, const int32_t* __restrict__ drafts,
    const int32_t* __restrict__ draft_len, int max_len, int vocab, int slice_len, int n_slices,
    Partial* __restrict__ partial, const int32_t* __restrict__ tree_parent,
    const int32_t* __restrict__ tree_len, int nodes) {
    constexpr int VW = (LT == DT_F32) ? 4 : 8;      // elements per 16-byte load
    constexpr int ES = (LT == DT_F32) ? 4 : 2;      // element size
    const int item = blockIdx.x;
    const int slice = blockIdx.y;
    const int tid = threadIdx.x;
    int64_t row = item;
    // The row's token and the loads that decide whether the row is judged
    // are requested together (every index is in range either way).
    const int tok = drafts[item];
    if constexpr (TREE) {
        const int g = item / nodes, u = item - g * nodes;
        const int tl = tree_len[g];
        const int par = tree_parent[item];
        if (u >= tl || par < -1 || par >= nodes) return;   // uniform over the block
        row = (int64_t)g * (nodes + 1) + 1 + par;
    } else {
        const int c = item / max_len, j = item - c * max_len;
        int len = draft_len ? draft_len[c] : max_len;
        len = len < 0 ? 0 : (len > max_len ? max_len : len);
        if (j >= len) return;                        // uniform over the block
    }

    const bool valid = tok >= 0 && tok < vocab;
    const char* rowp = (const char*)logits + row * row_stride * ES;
    const int tk = valid ? tok : -1;                 // -1: the count is unused

    const int v0 = slice * slice_len;
    const int v1 = (v0 + slice_len < vocab) ? v0 + slice_len : vocab;
    Acc acc;
    float mx = -__builtin_inff();
    __shared__ float s_max[kRowWaves];

    if constexpr (VEC) {
        const int nvec = (v1 - v0) / VW;
        const u32x4* vp = (const u32x4*)(rowp + (int64_t)v0 * ES);
        u32x4 buf[kNV];
#pragma unroll
        for (int k = 0; k < kNV; ++k) {
            const int i = tid + k * kRowThreads;
            buf[k] = (i < nvec) ? __builtin_nontemporal_load(vp + i) : u32x4{0u, 0u, 0u, 0u};
        }
        // Fewer than VW trailing elements (last slice only), and the judged
        // token's logit: both requested unconditionally (clamped to a real
        // element) together with the slice, so that no load waits for
        // another.
        const int vt = v0 + nvec * VW + tid;
        const bool has_t = vt < v1;
        const float xt_raw = load_one<LT>(rowp, has_t ? vt : v0);
        const float xd_raw = load_one<LT>(rowp, valid ? tok : v0);
        __builtin_amdgcn_sched_barrier(0);
        const float xt = has_t ? xt_raw : -__builtin_inff();
#pragma unroll
        for (int k = 0; k < kNV; ++k) {
            if (tid + k * kRowThreads < nvec) {
                float x[VW];
                unpack<LT>(buf[k], x);
#pragma unroll
                for (int u = 0; u < VW; ++u) mx = __builtin_fmaxf(mx, x[u]);
            }
        }
        mx = __builtin_fmaxf(mx, xt);
        const float wm = wave_max_f(mx);
        if ((tid & 63) == 0) s_max[tid >> 6] = wm;
        __syncthreads();
        const float m = waves_max(s_max);
        mx = m;
        // The thresholds of the rank count (left of d / from d on), formed
        // only here, so that the judged logit's load is not waited for
        // before phase 1.
        const float xd = valid ? xd_raw : 0.0f;
        const float thr_lo = xd, thr_hi = next_up(xd);
        {
            // An all -inf slice keeps weight 0 (t clamps) but still counts ties.
            const float nm = (m == -__builtin_inff()) ? 0.0f : -m * kLog2e;
            if (nvec >= kNV * kRowThreads) {
                // A full slice (every one but a row's last): no lane is
                // idle, so the rank count is a wave ballot per element,
                // counted on the scalar unit (one vector compare each).
                uint32_t wc = 0;
#pragma unroll
                for (int k = 0; k < kNV; ++k) {
                    const int i = tid + k * kRowThreads;
                    float x[VW];
                    unpack<LT>(buf[k], x);
                    const int vb = v0 + i * VW;
                    const float thr = (vb + VW <= tk) ? thr_lo : thr_hi;
#pragma unroll
                    for (int u = 0; u < VW; ++u) {
                        absorb_sum(acc, x[u], nm);
                        wc += (uint32_t)__popcll(__ballot(x[u] >= thr));
                    }
                }
                acc.wcnt = wc;
            } else {
#pragma unroll
                for (int k = 0; k < kNV; ++k) {
                    const int i = tid + k * kRowThreads;
                    if (i < nvec) {
                        float x[VW];
                        unpack<LT>(buf[k], x);
                        const int vb = v0 + i * VW;
                        const float thr = (vb + VW <= tk) ? thr_lo : thr_hi;
#pragma unroll
                        for (int u = 0; u < VW; ++u) absorb(acc, x[u], nm, thr);
                    }
                }
            }
            if (has_t) absorb(acc, xt, nm, vt < tk ? thr_lo : thr_hi);
            // The vector holding d was counted with x > x_d throughout; its
            // elements left of d equal to x_d also rank above d.  Only the
            // thread that holds it adds them (its registers, picked by
            // selects), so no other element pays for the test.
            const int id = (tk - v0) / VW;
            if (tk > v0 && id < nvec && id % kRowThreads == tid && tk - (v0 + id * VW) > 0) {
                const int kd = id / kRowThreads;
                u32x4 w = buf[0];
#pragma unroll
                for (int k = 1; k < kNV; ++k) w = (k == kd) ? buf[k] : w;
                float x[VW];
                unpack<LT>(w, x);
                const int nl = tk - (v0 + id * VW);
#pragma unroll
                for (int u = 0; u < VW; ++u) acc.cnt += (u < nl && x[u] == xd) ? 1 : 0;
            }
        }
    } else {
        // Unconditional loads (positions past the slice re-read its first
        // element and are set to -inf), so all of them are in flight at once.
        float x[kScalarPer];
#pragma unroll
        for (int k = 0; k < kScalarPer; ++k) {
            const int v = v0 + tid + k * kRowThreads;
            x[k] = load_one<LT>(rowp, v < v1 ? v : v0);
        }
        const float xd_raw = load_one<LT>(rowp, valid ? tok : v0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < kScalarPer; ++k) {
            const int v = v0 + tid + k * kRowThreads;
            if (v >= v1) x[k] = -__builtin_inff();
            mx = __builtin_fmaxf(mx, x[k]);
        }
        const float wm = wave_max_f(mx);
        if ((tid & 63) == 0) s_max[tid >> 6] = wm;
        __syncthreads();
        const float m = waves_max(s_max);
        mx = m;
        const float xd = valid ? xd_raw : 0.0f;
        const float thr_lo = xd, thr_hi = next_up(xd);   // left of d / from d on
        {
            const float nm = (m == -__builtin_inff()) ? 0.0f : -m * kLog2e;
#pragma unroll
            for (int k = 0; k < kScalarPer; ++k) {
                const int v = v0 + tid + k * kRowThreads;
                if (v < v1) absorb(acc, x[k], nm, v < tk ? thr_lo : thr_hi);
            }
        }
    }

    // Block sums in a fixed order.
    const float ws = wave_sum_f(acc.s), wt = wave_sum_f(acc.t2);
    const int wc = wave_sum_i(acc.cnt) + (int)acc.wcnt;
    __shared__ Partial s_w[kRowWaves];
    if ((tid & 63) == 0) s_w[tid >> 6] = Partial{mx, ws, wt, wc};
    __syncthreads();
    if (tid == 0) {
        Partial p{mx, pair_sum<kRowWaves, float>([&](int w) { return s_w[w].s; }, 0),
                  pair_sum<kRowWaves, float>([&](int w) { return s_w[w].t2; }, 0),
                  pair_sum<kRowWaves, int>([&](int w) { return s_w[w].cnt; }, 0)};
        partial[(int64_t)item * n_slices + slice] = p;
    }
}

constexpr int kFinThreads = 512;
constexpr int kFinChunkRows = 4096;   // (candidate, position) rows per LDS chunk
constexpr int kFinChunkCands = 1024;  // candidates per LDS chunk

__device__ __forceinline__ uint64_t bits_upto(int x) {  // bits 0..x set (x may be -1)
    return (x >= 63) ? ~0ull : ((x < 0) ? 0ull : ((1ull << (x + 1)) - 1ull));
}

// Merge of an item's slice partials in slice order.  Loads go out in
// batches of kMergeBatch (clamped indices, no branch around a load, so none
// waits for the one before it); the first merge with the empty state returns
// slice 0 unchanged.
constexpr int kMergeBatch = 8;

__device__ __forceinline__ void merge_partials(const Partial* p, int n_slices, Stats* st,
                                               int* cnt) {
    Stats a{-__builtin_inff(), 0.0f, 0.0f};
    int c = 0;
    for (int s0 = 0; s0 < n_slices; s0 += kMergeBatch) {
        Partial q[kMergeBatch];
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u)
            q[u] = p[(s0 + u < n_slices) ? s0 + u : n_slices - 1];
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
            if (s0 + u < n_slices) {
                a = (s0 + u == 0) ? Stats{q[u].m, q[u].s, q[u].t2}
                                  : merge(a, Stats{q[u].m, q[u].s, q[u].t2});
                c += q[u].cnt;
            }
        }
    }
    *st = a;
    *cnt = c;
}

// Row statistics of one item from its merged partials: the entropy score
// and the rank of the judged token; bits em | ent<<1 | topk<<2.
__device__ __forceinline__ uint8_t item_bits(const Stats& a, int cnt, int tok, int vocab,
                                             const GateParams& gp, float* score, int* rank) {
    const float e_nats = __logf(a.s) - (kLn2 * a.t2) / a.s;
    *score = e_nats * gp.ent_scale;
    const bool valid = tok >= 0 && tok < vocab;
    *rank = valid ? cnt : vocab;
    return (uint8_t)((valid && *rank == 0 ? 1 : 0) | (*score > gp.gamma ? 2 : 0) |
                     (valid && *rank < gp.topk ? 4 : 0));
}

// First candidate with the largest n in the block (all threads call it).
// A thread's (n, i) is one key, n + 1 above the complemented index, so the
// largest key has the largest n and then the smallest i (a thread that saw
// no candidate has n = -1, below every real one); each wave takes its
// maximum with lane swaps and thread 0 the waves'.
__device__ void group_best(int best_n, int best_i, int32_t* out) {
    __shared__ uint64_t s_w[kFinThreads / 64];
    uint64_t key = ((uint64_t)(uint32_t)(best_n + 1) << 32) |
                   (uint64_t)(0xFFFFFFFFu - (uint32_t)best_i);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint64_t o = __shfl_xor(key, off, 64);
        key = o > key ? o : key;
    }
    if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = key;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t m = s_w[0];
#pragma unroll
        for (int w = 1; w < kFinThreads / 64; ++w) m = s_w[w] > m ? s_w[w] : m;
        *out = (int32_t)(0xFFFFFFFFu - (uint32_t)m);
    }
}

// Dense finalize, one block per group, in chunks of candidates.  Phase 1
// gives every (candidate, position) row a thread: the row's bits into LDS
// and its exact-match bit into the candidate's 64-bit mask.  Phase 2 gives
// every row a thread again: the mismatches in its window from the mask (one
// popcount), its gate bit (Alg. 4's cascade) into the candidate's gate
// mask.  Phase 3 gives every candidate a thread: the leading run of the gate
// mask is the accepted length.  No thread walks a draft's positions, so the
// cost does not grow with the draft length.
__global__ __launch_bounds__(kFinThreads) void verify_finalize_kernel(
    const Partial* __restrict__ partial, int n_slices, const int32_t* __restrict__ drafts,
    const int32_t* __restrict__ draft_len, int max_len, int vocab, int group_size,
    GateParams gp, int32_t* __restrict__ out_accept_len, int32_t* __restrict__ out_best,
    float* __restrict__ out_gate_score, uint8_t* __restrict__ out_masks,
    int32_t* __restrict__ out_rank) {
    __shared__ uint8_t s_bits[kFinChunkRows];     // em | ent<<1 | topk<<2 per row
    __shared__ uint8_t s_len[kFinChunkCands];     // clamped draft length per candidate
    __shared__ uint64_t s_em[kFinChunkCands];     // exact-match bit per position
    __shared__ uint64_t s_gate[kFinChunkCands];   // gate bit per position
    const int g = blockIdx.x;
    const int by_rows = kFinChunkRows / max_len;
    const int chunk_cands = by_rows < kFinChunkCands ? by_rows : kFinChunkCands;
    const uint64_t in_draft = bits_upto(max_len - 1);
    for (int cl = threadIdx.x; cl < kFinChunkCands; cl += kFinThreads) {
        s_em[cl] = 0ull;
        s_gate[cl] = 0ull;
    }
    __syncthreads();
    int best_n = -1, best_i = 0;
    for (int cc0 = 0; cc0 < group_size; cc0 += chunk_cands) {
        const int ncc = (group_size - cc0 < chunk_cands) ? group_size - cc0 : chunk_cands;
        const int rows = ncc * max_len;
        // Phase 1: the row statistics.
        for (int r = threadIdx.x; r < rows; r += kFinThreads) {
            const int cl = r / max_len, jj = r - cl * max_len;
            const int c = g * group_size + cc0 + cl;
            const int64_t row = (int64_t)c * max_len + jj;
            // Every load of the row first (the partials of a position past
            // the draft were not written and are not used).
            int len = draft_len ? draft_len[c] : max_len;
            const int tok = drafts[row];
            Stats st;
            int cnt;
            merge_partials(partial + row * n_slices, n_slices, &st, &cnt);
            len = len < 0 ? 0 : (len > max_len ? max_len : len);
            uint8_t bits = 0;
            float score = 0.0f;
            int rank = vocab;
            if (jj < len) bits = item_bits(st, cnt, tok, vocab, gp, &score, &rank);
            if (out_gate_score) out_gate_score[row] = score;
            if (out_rank) out_rank[row] = rank;
            s_bits[r] = bits;
            if (jj == 0) s_len[cl] = (uint8_t)len;
            if (bits & 1) atomicOr((unsigned long long*)&s_em[cl], 1ull << jj);
        }
        __syncthreads();
        // Phase 2: each row's window and gate.  Mismatches are 1 - B_em
        // inside the draft (every position past its length included) and
        // W padding ones past the last position.
        for (int r = threadIdx.x; r < rows; r += kFinThreads) {
            const int cl = r / max_len, jj = r - cl * max_len;
            const uint8_t b = s_bits[r];
            const uint64_t notem = ~s_em[cl] & in_draft;
            const int hi = jj + gp.window;
            const int in_hi = hi < max_len - 1 ? hi : max_len - 1;
            const uint64_t range = bits_upto(in_hi) & ~bits_upto(jj);
            const int mis = __popcll(notem & range) + (hi > max_len - 1 ? hi - (max_len - 1) : 0);
            const bool con = mis <= gp.tau;
            const bool bem = b & 1, bent = (b >> 1) & 1, btk = (b >> 2) & 1;
            const bool gate = (jj < (int)s_len[cl]) && (bem || (bent && (btk || con)));
            if (out_masks) {
                const int64_t row = (int64_t)(g * group_size + cc0 + cl) * max_len + jj;
                out_masks[row] = (uint8_t)((int)bem | ((int)bent << 1) | ((int)btk << 2) |
                                           ((int)con << 3) | ((int)gate << 4));
            }
            if (gate) atomicOr((unsigned long long*)&s_gate[cl], 1ull << jj);
        }
        __syncthreads();
        // Phase 3: the accepted length, and the masks cleared for the next
        // chunk (each candidate's words by its own thread).
        for (int cl = threadIdx.x; cl < ncc; cl += kFinThreads) {
            const uint64_t open = ~s_gate[cl];
            const int n = open == 0ull ? 64 : __builtin_ctzll(open);
            out_accept_len[g * group_size + cc0 + cl] = n;
            if (n > best_n) {
                best_n = n;
                best_i = cc0 + cl;
            }
            s_em[cl] = 0ull;
            s_gate[cl] = 0ull;
        }
        __syncthreads();
    }
    group_best(best_n, best_i, out_best + g);
}

// Tree variant, one block per group.  Phase 1 gives every tree node of the
// group a thread (bits, score and rank into LDS).  Then every (draft,
// position) row gets a thread in three phases: its node through Gamma and
// whether that node is judged (into the draft's 64-bit mask); the draft's
// length, the leading run of that mask, and the row's bits and outputs
// (exact-match bit into the draft's mask); its window and gate bit, as in
// the dense finalize.  Last, every draft a thread for the leading run of its
// gate mask.
__global__ __launch_bounds__(kFinThreads) void verify_finalize_tree_kernel(
    const Partial* __restrict__ partial, int n_slices, const int32_t* __restrict__ tree_tokens,
    const int32_t* __restrict__ tree_parent, const int32_t* __restrict__ tree_len,
    const int32_t* __restrict__ gamma, int max_len, int vocab, int group_size, GateParams gp,
    int32_t* __restrict__ out_accept_len, int32_t* __restrict__ out_best,
    float* __restrict__ out_gate_score, uint8_t* __restrict__ out_masks,
    int32_t* __restrict__ out_rank) {
    __shared__ uint8_t s_bits[kMaxNodes];       // em | ent<<1 | topk<<2 | judged<<3 per node
    __shared__ float s_score[kMaxNodes];
    __shared__ int32_t s_rank[kMaxNodes];
    __shared__ int16_t s_node[kMaxNodes];       // per row: its judged node, else -1
    __shared__ uint8_t s_rbits[kMaxNodes];      // per row: its node's bits inside the draft
    __shared__ uint64_t s_run[kMaxGroup];       // per draft: positions with a judged node
    __shared__ uint64_t s_em[kMaxGroup];        // per draft: exact-match bits
    __shared__ uint64_t s_gate[kMaxGroup];      // per draft: gate bits
    __shared__ uint8_t s_len[kMaxGroup];        // per draft: its length
    const int g = blockIdx.x;
    const int nodes = group_size * max_len;
    const int L = tree_len[g] < nodes ? tree_len[g] : nodes;
    const uint64_t in_draft = bits_upto(max_len - 1);
    for (int cl = threadIdx.x; cl < group_size; cl += kFinThreads) {
        s_run[cl] = 0ull;
        s_em[cl] = 0ull;
        s_gate[cl] = 0ull;
    }
    for (int u = threadIdx.x; u < L; u += kFinThreads) {
        const int item = g * nodes + u;
        // Every load of the node first (the partials of a node that is not
        // judged were not written and are not used).
        const int tok = tree_tokens[item];
        const int par = tree_parent[item];
        Stats st;
        int cnt;
        merge_partials(partial + (int64_t)item * n_slices, n_slices, &st, &cnt);
        uint8_t bits = 0;
        float score = 0.0f;
        int rank = vocab;
        // u < L: the node exists; it is judged when its parent is in range
        // (the rows kernel's test for the same node).
        if (par >= -1 && par < nodes) bits = 8 | item_bits(st, cnt, tok, vocab, gp, &score, &rank);
        s_bits[u] = bits;
        s_score[u] = score;
        s_rank[u] = rank;
    }
    __syncthreads();
    // Rows: the node of each draft position, and whether it is judged.
    for (int r = threadIdx.x; r < nodes; r += kFinThreads) {
        const int cl = r / max_len, jj = r - cl * max_len;
        const int u = gamma[(int64_t)(g * group_size + cl) * max_len + jj];
        const bool judged = u >= 0 && u < L && (s_bits[u] & 8);
        s_node[r] = judged ? (int16_t)u : (int16_t)-1;
        if (judged) atomicOr((unsigned long long*)&s_run[cl], 1ull << jj);
    }
    __syncthreads();
    // Rows: a draft's length is its leading run of judged positions; the
    // bits and outputs of the positions inside it.
    for (int r = threadIdx.x; r < nodes; r += kFinThreads) {
        const int cl = r / max_len, jj = r - cl * max_len;
        const uint64_t unjudged = ~s_run[cl];
        const int len = unjudged == 0ull ? 64 : __builtin_ctzll(unjudged);
        const bool inside = jj < len;
        const int u = s_node[r];
        const uint8_t b = inside ? s_bits[u] : 0;
        const int64_t o = (int64_t)(g * group_size + cl) * max_len + jj;
        if (out_gate_score) out_gate_score[o] = inside ? s_score[u] : 0.0f;
        if (out_rank) out_rank[o] = inside ? s_rank[u] : vocab;
        s_rbits[r] = b;
        if (jj == 0) s_len[cl] = (uint8_t)len;
        if (b & 1) atomicOr((unsigned long long*)&s_em[cl], 1ull << jj);
    }
    __syncthreads();
    // Rows: window and gate.
    for (int r = threadIdx.x; r < nodes; r += kFinThreads) {
        const int cl = r / max_len, jj = r - cl * max_len;
        const uint8_t b = s_rbits[r];
        const uint64_t notem = ~s_em[cl] & in_draft;
        const int hi = jj + gp.window;
        const int in_hi = hi < max_len - 1 ? hi : max_len - 1;
        const uint64_t range = bits_upto(in_hi) & ~bits_upto(jj);
        const int mis = __popcll(notem & range) + (hi > max_len - 1 ? hi - (max_len - 1) : 0);
        const bool con = mis <= gp.tau;
        const bool bem = b & 1, bent = (b >> 1) & 1, btk = (b >> 2) & 1;
        const bool gate = (jj < (int)s_len[cl]) && (bem || (bent && (btk || con)));
        if (out_masks) {
            const int64_t o = (int64_t)(g * group_size + cl) * max_len + jj;
            out_masks[o] = (uint8_t)((int)bem | ((int)bent << 1) | ((int)btk << 2) |
                                     ((int)con << 3) | ((int)gate << 4));
        }
        if (gate) atomicOr((unsigned long long*)&s_gate[cl], 1ull << jj);
    }
    __syncthreads();
    int best_n = -1, best_i = 0;
    for (int cl = threadIdx.x; cl < group_size; cl += kFinThreads) {
        const uint64_t open = ~s_gate[cl];
        const int n = open == 0ull ? 64 : __builtin_ctzll(open);
        out_accept_len[g * group_size + cl] = n;
        if (n > best_n) {
            best_n = n;
            best_i = cl;
        }
    }
    group_best(best_n, best_i, out_best + g);
}

struct Plan {
    bool vec;
    int n_slices;
    int slice_len;
};

Plan plan_slices(int vocab, int dtype, bool vec) {
    const int vw = (dtype == DT_F32) ? 4 : 8;
    const int slice_len = vec ? kRowThreads * kNV * vw : kRowThreads * kScalarPer;
    return Plan{vec, (vocab + slice_len - 1) / slice_len, slice_len};
}

template <int LT, bool TREE>
hipError_t launch_rows_t(const void* logits, int64_t row_stride, const int32_t* tokens,
                         const int32_t* draft_len, int64_t n_items, int max_len, int vocab,
                         const Plan& pl, Partial* part, const int32_t* tree_parent,
                         const int32_t* tree_len, int nodes, hipStream_t stream) {
    const dim3 grid((unsigned)n_items, (unsigned)pl.n_slices);
    if (pl.vec)
        hipLaunchKernelGGL((verify_rows_kernel<LT, true, TREE>), grid, dim3(kRowThreads), 0,
                           stream, logits, row_stride, tokens, draft_len, max_len, vocab,
                           pl.slice_len, pl.n_slices, part, tree_parent, tree_len, nodes);
    else
        hipLaunchKernelGGL((verify_rows_kernel<LT, false, TREE>), grid, dim3(kRowThreads), 0,
                           stream, logits, row_stride, tokens, draft_len, max_len, vocab,
                           pl.slice_len, pl.n_slices, part, tree_parent, tree_len, nodes);
    return hipGetLastError();
}

template <bool TREE>
hipError_t launch_rows(const void* logits, int logits_dtype, int64_t row_stride,
                       const int32_t* tokens, const int32_t* draft_len, int64_t n_items,
                       int max_len, int vocab, const Plan& pl, Partial* part,
                       const int32_t* tree_parent, const int32_t* tree_len, int nodes,
                       hipStream_t stream) {
    switch (logits_dtype) {
        case DT_F32:
            return launch_rows_t<DT_F32, TREE>(logits, row_stride, tokens, draft_len, n_items,
                                               max_len, vocab, pl, part, tree_parent, tree_len,
                                               nodes, stream);
        case DT_F16:
            return launch_rows_t<DT_F16, TREE>(logits, row_stride, tokens, draft_len, n_items,
                                               max_len, vocab, pl, part, tree_parent, tree_len,
                                               nodes, stream);
        default:
            return launch_rows_t<DT_BF16, TREE>(logits, row_stride, tokens, draft_len, n_items,
                                                max_len, vocab, pl, part, tree_parent, tree_len,
                                                nodes, stream);
    }
}

Plan make_plan(const void* logits, int logits_dtype, int64_t row_stride, int vocab) {
    const int es = (logits_dtype == DT_F32) ? 4 : 2;
    const bool vec = ((uintptr_t)logits % 16 == 0) && ((row_stride * es) % 16 == 0);
    return plan_slices(vocab, logits_dtype, vec);
}

}  // namespace

size_t verify_workspace_bytes(int n_cand, int max_len, int vocab) {
    // The unaligned-row plan has the most slices.
    const Plan p = plan_slices(vocab, DT_BF16, false);
    return (size_t)n_cand * (size_t)max_len * (size_t)p.n_slices * sizeof(Partial);
}

size_t verify_tree_workspace_bytes(int n_cand, int max_len, int vocab, int n_groups) {
    // One partial per (tree node, slice); a group has at most n_cand / n_groups
    // * max_len nodes, so the dense bound is also the tree bound.
    (void)n_groups;
    return verify_workspace_bytes(n_cand, max_len, vocab);
}

hipError_t launch_verify(const void* logits, int logits_dtype, int64_t row_stride,
                         const int32_t* drafts, const int32_t* draft_len, int n_cand,
                         int max_len, int vocab, int n_groups, const GateParams& gp,
                         int32_t* out_accept_len, int32_t* out_best, float* out_gate_score,
                         uint8_t* out_masks, int32_t* out_rank, void* workspace,
                         hipStream_t stream) {
    if (n_cand == 0) return hipSuccess;
    const Plan pl = make_plan(logits, logits_dtype, row_stride, vocab);
    Partial* part = (Partial*)workspace;
    hipError_t e = launch_rows<false>(logits, logits_dtype, row_stride, drafts, draft_len,
                                      (int64_t)n_cand * max_len, max_len, vocab, pl, part,
                                      nullptr, nullptr, 0, stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(verify_finalize_kernel, dim3((unsigned)n_groups), dim3(kFinThreads), 0,
                       stream, part, pl.n_slices, drafts, draft_len, max_len, vocab,
                       n_cand / n_groups, gp, out_accept_len, out_best, out_gate_score,
                       out_masks, out_rank);
    return hipGetLastError();
}

hipError_t launch_verify_tree(const void* logits, int logits_dtype, int64_t row_stride,
                              const int32_t* tree_tokens, const int32_t* tree_parent,
                              const int32_t* tree_len, const int32_t* gamma, int n_cand,
                              int max_len, int vocab, int n_groups, const GateParams& gp,
                              int32_t* out_accept_len, int32_t* out_best, float* out_gate_score,
                              uint8_t* out_masks, int32_t* out_rank, void* workspace,
                              hipStream_t stream) {
    if (n_cand == 0) return hipSuccess;
    const Plan pl = make_plan(logits, logits_dtype, row_stride, vocab);
    Partial* part = (Partial*)workspace;
    const int gs = n_cand / n_groups;
    const int nodes = gs * max_len;
    hipError_t e = launch_rows<true>(logits, logits_dtype, row_stride, tree_tokens, nullptr,
                                     (int64_t)n_groups * nodes, max_len, vocab, pl, part,
                                     tree_parent, tree_len, nodes, stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(verify_finalize_tree_kernel, dim3((unsigned)n_groups), dim3(kFinThreads),
                       0, stream, part, pl.n_slices, tree_tokens, tree_parent, tree_len, gamma,
                       max_len, vocab, gs, gp, out_accept_len, out_best, out_gate_score,
                       out_masks, out_rank);
    return hipGetLastError();
}

}  // namespace sense
