// Soft-gated evaluation (Sec. 3.3 Eqs. 12-18; Alg. 4) of a candidate draft
// batch against the target's aligned logits.
//
// The cost is one read of the logits of every live (candidate, position)
// row; everything else is per-row scalars.  Two kernels:
//
// verify_rows: one block of 256 threads per (row, vocabulary slice).  Each
//   thread streams its part of the slice with 16-byte loads and keeps, in
//   one pass,
//     m   running maximum,
//     S   sum of 2^(t) with t = (x - m) log2 e     (= sum e^(x-m)),
//     T2  sum of 2^(t) * t                          (= log2 e * sum e^(x-m)(x-m)),
//     cnt #{v : x_v > x_d} + #{v < d : x_v = x_d},  x_d the draft token's logit,
//   rescaling S and T2 when the maximum grows.  The block merges its 256
//   states (DPP butterflies in a fixed order, then the four waves in order)
//   and stores one 16-byte partial per (row, slice).  With p = softmax(x),
//   E = -sum p ln p = ln S - ln2 * T2 / S.  The draft token is the first
//   argmax exactly when cnt = 0, and it is in the top-k set exactly when
//   cnt < k, so neither an argmax nor a sort of the vocabulary is needed.
//   Slices exist only to give small batches enough blocks.
//
// verify_finalize: one block per candidate group.  Each thread takes a
//   candidate, merges the slices of its rows in slice order, forms the
//   masks, counts window mismatches with a popcount over 64-bit masks, finds
//   the leading run of accepted positions, and the block picks the group's
//   first longest candidate.
#include "internal.h"

namespace sense {
namespace {

constexpr int kRowThreads = 256;
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

// Merge of two (m, S, T2) states; symmetric in its arguments bit for bit.
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
__device__ __forceinline__ float dpp_f(float x) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
    return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ void butterfly_step(Stats& st, int& cnt) {
    Stats o{dpp_f<CTRL>(st.m), dpp_f<CTRL>(st.s), dpp_f<CTRL>(st.t2)};
    st = merge(st, o);
    cnt += dpp_i<CTRL>(cnt);
}
__device__ __forceinline__ Stats lane_read(const Stats& st, int lane) {
    return Stats{__builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, st.m), lane)),
                 __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, st.s), lane)),
                 __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, st.t2), lane))};
}

template <int LT>
__device__ __forceinline__ float load_one(const void* base, int64_t i) {
    if constexpr (LT == DT_F32) {
        return ((const float*)base)[i];
    } else if constexpr (LT == DT_BF16) {
        return __builtin_bit_cast(float, (uint32_t)((const uint16_t*)base)[i] << 16);
    } else {
        return (float)__builtin_bit_cast(_Float16, ((const uint16_t*)base)[i]);
    }
}

struct RowState {
    float m, nm, s, t2;  // nm = -m * log2 e
    int cnt;
};

__device__ __forceinline__ void absorb_max(RowState& st, float vmax) {
    if (vmax > st.m) {
        if (st.m == -__builtin_inff()) {
            st.s = 0.0f;
            st.t2 = 0.0f;
        } else {
            const float dl = (st.m - vmax) * kLog2e;
            const float a = fast_exp2(dl);
            st.t2 = a * __builtin_fmaf(dl, st.s, st.t2);
            st.s = a * st.s;
        }
        st.m = vmax;
        st.nm = -vmax * kLog2e;
    }
}

__device__ __forceinline__ void absorb(RowState& st, float x, int v, float xd, int tok) {
    // The clamp keeps a -inf logit at weight 0 and contribution 0 (not 0*inf).
    const float t = __builtin_fmaxf(__builtin_fmaf(x, kLog2e, st.nm), -256.0f);
    const float e = fast_exp2(t);
    st.s += e;
    st.t2 = __builtin_fmaf(e, t, st.t2);
    st.cnt += (x > xd) | ((x == xd) & (v < tok));
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

template <int LT, bool VEC>
__global__ __launch_bounds__(kRowThreads) void verify_rows_kernel(
    const void* __restrict__ logits, int64_t row_stride, const int32_t* __restrict__ drafts,
    const int32_t* __restrict__ draft_len, int max_len, int vocab, int slice_len, int n_slices,
    Partial* __restrict__ partial) {
    constexpr int VW = (LT == DT_F32) ? 4 : 8;      // elements per 16-byte load
    constexpr int ES = (LT == DT_F32) ? 4 : 2;      // element size
    const int row = blockIdx.x;
    const int slice = blockIdx.y;
    const int c = row / max_len, j = row - c * max_len;
    int len = draft_len ? draft_len[c] : max_len;
    len = len < 0 ? 0 : (len > max_len ? max_len : len);
    if (j >= len) return;

    const int tok = drafts[row];
    const bool valid = tok >= 0 && tok < vocab;
    const char* rowp = (const char*)logits + (int64_t)row * row_stride * ES;
    const float xd = valid ? load_one<LT>(rowp, tok) : 0.0f;
    const int tk = valid ? tok : -1;   // with tk = -1 and xd = 0 the count is unused

    const int v0 = slice * slice_len;
    const int v1 = (v0 + slice_len < vocab) ? v0 + slice_len : vocab;
    RowState st{-__builtin_inff(), 0.0f, 0.0f, 0.0f, 0};

    int vtail = v0;
    if constexpr (VEC) {
        const int nvec = (v1 - v0) / VW;
        const u32x4* vp = (const u32x4*)(rowp + (int64_t)v0 * ES);
        for (int i = threadIdx.x; i < nvec; i += kRowThreads) {
            const u32x4 w = __builtin_nontemporal_load(vp + i);
            float x[VW];
            unpack<LT>(w, x);
            float vmax = x[0];
#pragma unroll
            for (int u = 1; u < VW; ++u) vmax = x[u] > vmax ? x[u] : vmax;
            absorb_max(st, vmax);
            const int vb = v0 + i * VW;
#pragma unroll
            for (int u = 0; u < VW; ++u) absorb(st, x[u], vb + u, xd, tk);
        }
        vtail = v0 + nvec * VW;
    }
    for (int v = vtail + threadIdx.x; v < v1; v += kRowThreads) {
        const float x = load_one<LT>(rowp, v);
        absorb_max(st, x);
        absorb(st, x, v, xd, tk);
    }

    // Block merge: butterflies inside each 16-lane row, rows in order, waves
    // in order.
    Stats s{st.m, st.s, st.t2};
    int cnt = st.cnt;
    butterfly_step<0xB1>(s, cnt);
    butterfly_step<0x4E>(s, cnt);
    butterfly_step<0x141>(s, cnt);
    butterfly_step<0x140>(s, cnt);
    Stats w = merge(merge(lane_read(s, 0), lane_read(s, 16)),
                    merge(lane_read(s, 32), lane_read(s, 48)));
    const int wc = __builtin_amdgcn_readlane(cnt, 0) + __builtin_amdgcn_readlane(cnt, 16) +
                   __builtin_amdgcn_readlane(cnt, 32) + __builtin_amdgcn_readlane(cnt, 48);
    __shared__ Partial s_w[kRowThreads / 64];
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) s_w[wave] = Partial{w.m, w.s, w.t2, wc};
    __syncthreads();
    if (threadIdx.x == 0) {
        Stats a{s_w[0].m, s_w[0].s, s_w[0].t2};
        int tc = s_w[0].cnt;
#pragma unroll
        for (int i = 1; i < kRowThreads / 64; ++i) {
            a = merge(a, Stats{s_w[i].m, s_w[i].s, s_w[i].t2});
            tc += s_w[i].cnt;
        }
        partial[(int64_t)row * n_slices + slice] = Partial{a.m, a.s, a.t2, tc};
    }
}

constexpr int kFinThreads = 256;

__device__ __forceinline__ uint64_t bits_upto(int x) {  // bits 0..x set (x may be -1)
    return (x >= 63) ? ~0ull : ((x < 0) ? 0ull : ((1ull << (x + 1)) - 1ull));
}

__global__ __launch_bounds__(kFinThreads) void verify_finalize_kernel(
    const Partial* __restrict__ partial, int n_slices, const int32_t* __restrict__ drafts,
    const int32_t* __restrict__ draft_len, int max_len, int vocab, int group_size,
    GateParams gp, int32_t* __restrict__ out_accept_len, int32_t* __restrict__ out_best,
    float* __restrict__ out_gate_score, uint8_t* __restrict__ out_masks,
    int32_t* __restrict__ out_rank) {
    const int g = blockIdx.x;
    int best_n = -1, best_i = 0;
    for (int cc = threadIdx.x; cc < group_size; cc += kFinThreads) {
        const int c = g * group_size + cc;
        int len = draft_len ? draft_len[c] : max_len;
        len = len < 0 ? 0 : (len > max_len ? max_len : len);
        uint64_t em = 0, ent = 0, tkm = 0;
        for (int j = 0; j < len; ++j) {
            const int64_t row = (int64_t)c * max_len + j;
            const Partial* p = partial + row * n_slices;
            Stats a{p[0].m, p[0].s, p[0].t2};
            int cnt = p[0].cnt;
            for (int s = 1; s < n_slices; ++s) {
                a = merge(a, Stats{p[s].m, p[s].s, p[s].t2});
                cnt += p[s].cnt;
            }
            const float e_nats = __logf(a.s) - (kLn2 * a.t2) / a.s;
            const float score = e_nats * gp.ent_scale;
            const int tok = drafts[row];
            const bool valid = tok >= 0 && tok < vocab;
            const int rank = valid ? cnt : vocab;
            if (valid && rank == 0) em |= 1ull << j;
            if (score > gp.gamma) ent |= 1ull << j;
            if (valid && rank < gp.topk) tkm |= 1ull << j;
            if (out_gate_score) out_gate_score[row] = score;
            if (out_rank) out_rank[row] = rank;
        }
        // Mismatches: 1 - B_em inside the draft, and W padding ones after it.
        const uint64_t notem = ~em & bits_upto(max_len - 1);
        int n = 0;
        bool still = true;
        for (int j = 0; j < max_len; ++j) {
            const int hi = j + gp.window;
            const int in_hi = hi < max_len - 1 ? hi : max_len - 1;
            const uint64_t range = bits_upto(in_hi) & ~bits_upto(j);
            const int r = __popcll(notem & range) + (hi > max_len - 1 ? hi - (max_len - 1) : 0);
            const bool con = r <= gp.tau;
            const bool bem = (em >> j) & 1, bent = (ent >> j) & 1, btk = (tkm >> j) & 1;
            const bool gate = (j < len) && (bem || (bent && (btk || con)));
            if (still && gate) ++n; else still = false;
            const int64_t row = (int64_t)c * max_len + j;
            if (out_masks)
                out_masks[row] = (uint8_t)((int)bem | ((int)bent << 1) | ((int)btk << 2) |
                                           ((int)con << 3) | ((int)gate << 4));
            if (j >= len) {
                if (out_gate_score) out_gate_score[row] = 0.0f;
                if (out_rank) out_rank[row] = vocab;
            }
        }
        out_accept_len[c] = n;
        if (n > best_n) {
            best_n = n;
            best_i = cc;
        }
    }
    // First candidate with the largest n in the group.
    __shared__ int s_n[kFinThreads], s_i[kFinThreads];
    s_n[threadIdx.x] = best_n;
    s_i[threadIdx.x] = best_i;
    __syncthreads();
    for (int off = kFinThreads / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            const int on = s_n[threadIdx.x + off], oi = s_i[threadIdx.x + off];
            if (on > s_n[threadIdx.x] || (on == s_n[threadIdx.x] && oi < s_i[threadIdx.x])) {
                s_n[threadIdx.x] = on;
                s_i[threadIdx.x] = oi;
            }
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) out_best[g] = s_i[0];
}

struct Plan {
    int n_slices;
    int slice_len;
};

Plan plan_slices(int n_cand, int max_len, int vocab, int dtype) {
    const int vw = (dtype == DT_F32) ? 4 : 8;
    const int64_t rows = (int64_t)n_cand * max_len;
    const int unit = kRowThreads * vw;                 // one vector per thread
    int max_slices = vocab / (4 * unit);               // >= 4 vectors per thread
    if (max_slices < 1) max_slices = 1;
    int64_t want = rows > 0 ? (2048 + rows - 1) / rows : 1;
    int ns = (int)(want < max_slices ? want : max_slices);
    if (ns < 1) ns = 1;
    int slice_len = (vocab + ns - 1) / ns;
    slice_len = (slice_len + unit - 1) / unit * unit;  // multiple of the vector width
    ns = (vocab + slice_len - 1) / slice_len;
    return Plan{ns, slice_len};
}

template <int LT>
hipError_t launch_rows(const void* logits, int64_t row_stride, const int32_t* drafts,
                       const int32_t* draft_len, int n_cand, int max_len, int vocab,
                       const Plan& pl, Partial* part, hipStream_t stream) {
    constexpr int ES = (LT == DT_F32) ? 4 : 2;
    const bool vec = ((uintptr_t)logits % 16 == 0) && ((row_stride * ES) % 16 == 0);
    const dim3 grid((unsigned)((int64_t)n_cand * max_len), (unsigned)pl.n_slices);
    if (vec)
        hipLaunchKernelGGL((verify_rows_kernel<LT, true>), grid, dim3(kRowThreads), 0, stream,
                           logits, row_stride, drafts, draft_len, max_len, vocab, pl.slice_len,
                           pl.n_slices, part);
    else
        hipLaunchKernelGGL((verify_rows_kernel<LT, false>), grid, dim3(kRowThreads), 0, stream,
                           logits, row_stride, drafts, draft_len, max_len, vocab, pl.slice_len,
                           pl.n_slices, part);
    return hipGetLastError();
}

}  // namespace

size_t verify_workspace_bytes(int n_cand, int max_len, int vocab) {
    // Sized for the widest plan (fp32 and 16-bit logits give the same or
    // fewer slices than this bound).
    const Plan a = plan_slices(n_cand, max_len, vocab, DT_F32);
    const Plan b = plan_slices(n_cand, max_len, vocab, DT_BF16);
    const int ns = a.n_slices > b.n_slices ? a.n_slices : b.n_slices;
    return (size_t)n_cand * (size_t)max_len * (size_t)ns * sizeof(Partial);
}

hipError_t launch_verify(const void* logits, int logits_dtype, int64_t row_stride,
                         const int32_t* drafts, const int32_t* draft_len, int n_cand,
                         int max_len, int vocab, int n_groups, const GateParams& gp,
                         int32_t* out_accept_len, int32_t* out_best, float* out_gate_score,
                         uint8_t* out_masks, int32_t* out_rank, void* workspace,
                         hipStream_t stream) {
    if (n_cand == 0) return hipSuccess;
    const Plan pl = plan_slices(n_cand, max_len, vocab, logits_dtype);
    Partial* part = (Partial*)workspace;
    hipError_t e;
    switch (logits_dtype) {
        case DT_F32:
            e = launch_rows<DT_F32>(logits, row_stride, drafts, draft_len, n_cand, max_len,
                                    vocab, pl, part, stream);
            break;
        case DT_F16:
            e = launch_rows<DT_F16>(logits, row_stride, drafts, draft_len, n_cand, max_len,
                                    vocab, pl, part, stream);
            break;
        default:
            e = launch_rows<DT_BF16>(logits, row_stride, drafts, draft_len, n_cand, max_len,
                                     vocab, pl, part, stream);
            break;
    }
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(verify_finalize_kernel, dim3((unsigned)n_groups), dim3(kFinThreads), 0,
                       stream, part, pl.n_slices, drafts, draft_len, max_len, vocab,
                       n_cand / n_groups, gp, out_accept_len, out_best, out_gate_score,
                       out_masks, out_rank);
    return hipGetLastError();
}

}  // namespace sense
