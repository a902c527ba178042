// Inverted-file retrieval: the approximate nearest-neighbour search that
// the paper runs through FAISS (Sec. 3.2 Eq. 7; App. implementation details:
// IVF-PQ, nlist 4096, nprobe 32, pq_m 16 on the 64-dim projected keys),
// here as IVF-Flat (exact scores inside the probed lists) and IVF-PQ
// (asymmetric distance computation on product-quantised residuals).
//
// Build (datastore construction, not the per-step path):
//   ivf_assign: every key's list = its most similar centroid (one thread per
//     key, the key in registers, centroids streamed through LDS in tiles);
//   pq_encode: code j of key i = nearest codebook entry of the residual
//     slice (one thread per key, all codebooks in LDS);
//   the index stores each list's rows contiguously (a counting sort by list:
//     histogram, exclusive scan, scatter); the order inside a list does not
//     enter any result, since candidates carry their original row id.
// Search (per step), for Q queries:
//   ivf_coarse: query-centroid similarities (probe ranking) and, for PQ, the
//     inner product of the (normalised) query with each centroid;
//   the probes = per-query top-nprobe of the coarse scores (the retrieval
//     top-k kernels);
//   ivf_scan_flat / ivf_scan_pq: blocks per query take its probes in turn;
//     each block finds where its probes' candidates start (exclusive prefix
//     of the probed list sizes in probe order; one block also stores the
//     query's candidate count), the PQ blocks build the query's tables
//     LUT[j][c] = u_j . C_j[c] in LDS, and each list's rows are scored into
//     packed (score, original row) keys;
//   the top-k kernels then select the k best keys per query and gather
//     their continuations.
#include "internal.h"

namespace sense {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kIvfThreads = 256;
constexpr int kAssignTile = 64;   // centroids per LDS tile in ivf_assign

__device__ __forceinline__ float wsum(float x) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) x += __shfl_xor(x, off, 64);
    return x;
}

__device__ __forceinline__ float key_elem(const uint16_t* row, int t, int dt) {
    const uint16_t b = row[t];
    if (dt == DT_F16) return (float)__builtin_bit_cast(_Float16, b);
    return __builtin_bit_cast(float, (uint32_t)b << 16);
}

// out_list[i] = argmax_l sim(key i, centroid l); ties to the lower l.
template <int KD>
__global__ __launch_bounds__(kIvfThreads) void ivf_assign_kernel(
    const uint16_t* __restrict__ keys, int key_dtype, int64_t n, int d, int64_t ld,
    const float* __restrict__ centroids, int nlist, int cosine, int32_t* __restrict__ out_list) {
    __shared__ float s_c[kAssignTile * KD];
    __shared__ float s_inv[kAssignTile];
    const int64_t i = (int64_t)blockIdx.x * kIvfThreads + threadIdx.x;
    float x[KD];
    float xn = 0.0f;
#pragma unroll
    for (int t = 0; t < KD; ++t) {
        x[t] = (i < n && t < d) ? key_elem(keys + i * ld, t, key_dtype) : 0.0f;
        xn = __builtin_fmaf(x[t], x[t], xn);
    }
    const float inv_x = (xn > 0.0f) ? 1.0f / __builtin_sqrtf(xn) : 0.0f;
    float best = -__builtin_inff();
    int arg = 0;
    for (int l0 = 0; l0 < nlist; l0 += kAssignTile) {
        const int nt = (nlist - l0 < kAssignTile) ? nlist - l0 : kAssignTile;
        __syncthreads();
        for (int e = threadIdx.x; e < nt * KD; e += kIvfThreads) {
            const int l = e / KD, t = e - l * KD;
            s_c[e] = t < d ? centroids[(int64_t)(l0 + l) * d + t] : 0.0f;
        }
        __syncthreads();
        if (cosine) {
            for (int l = threadIdx.x; l < nt; l += kIvfThreads) {
                float cn = 0.0f;
                for (int t = 0; t < d; ++t) cn = __builtin_fmaf(s_c[l * KD + t], s_c[l * KD + t], cn);
                s_inv[l] = (cn > 0.0f) ? 1.0f / __builtin_sqrtf(cn) : 0.0f;
            }
            __syncthreads();
        }
        for (int l = 0; l < nt; ++l) {
            float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
            for (int t = 0; t < KD; t += 2) {
                a0 = __builtin_fmaf(x[t], s_c[l * KD + t], a0);
                a1 = __builtin_fmaf(x[t + 1], s_c[l * KD + t + 1], a1);
            }
            float s = a0 + a1;
            if (cosine) s = (s * s_inv[l]) * inv_x;
            if (s > best) {
                best = s;
                arg = l0 + l;
            }
        }
    }
    if (i < n) out_list[i] = arg;
}

// Codes of key i: nearest codebook entry (squared L2, ties to the lower
// entry) to each slice of the residual key - centroid[list].  One thread per
// key; the residual slice (dsub <= kMaxDsub values) is formed when needed.
__global__ __launch_bounds__(kIvfThreads) void pq_encode_kernel(
    const uint16_t* __restrict__ keys, int key_dtype, int64_t n, int d, int64_t ld,
    const float* __restrict__ centroids, const int32_t* __restrict__ list_ids,
    const float* __restrict__ codebooks, int m, int ksub, int nlist,
    uint8_t* __restrict__ codes) {
    extern __shared__ float s_cb[];   // m * ksub * dsub = ksub * d floats
    for (int e = threadIdx.x; e < ksub * d; e += kIvfThreads) s_cb[e] = codebooks[e];
    __syncthreads();
    const int64_t i = (int64_t)blockIdx.x * kIvfThreads + threadIdx.x;
    if (i >= n) return;
    const int dsub = d / m;
    const int32_t li = list_ids[i];
    if (li < 0 || li >= nlist) {                 // no such list: code 0 throughout
        for (int j = 0; j < m; ++j) codes[i * m + j] = 0;
        return;
    }
    const float* c = centroids + (int64_t)li * d;
    const uint16_t* row = keys + i * ld;
    for (int j = 0; j < m; ++j) {
        float rs[kMaxDsub];
#pragma unroll
        for (int t = 0; t < kMaxDsub; ++t)
            rs[t] = t < dsub ? key_elem(row, j * dsub + t, key_dtype) - c[j * dsub + t] : 0.0f;
        float bd = __builtin_inff();
        int be = 0;
        for (int e = 0; e < ksub; ++e) {
            const float* cb = s_cb + ((int64_t)j * ksub + e) * dsub;
            float dist = 0.0f;
#pragma unroll
            for (int t = 0; t < kMaxDsub; ++t) {
                if (t < dsub) {
                    const float df = rs[t] - cb[t];
                    dist = __builtin_fmaf(df, df, dist);
                }
            }
            if (dist < bd) {
                bd = dist;
                be = e;
            }
        }
        codes[i * m + j] = (uint8_t)be;
    }
}

// inv[l] = 1 / ||row l|| of an fp32 matrix (0 for a zero row), one wave per row.
__global__ __launch_bounds__(kIvfThreads) void f32_inv_norm_kernel(const float* __restrict__ rows,
                                                                   int n, int d,
                                                                   float* __restrict__ inv) {
    const int lane = threadIdx.x & 63;
    const int r = blockIdx.x * (kIvfThreads / 64) + (threadIdx.x >> 6);
    if (r >= n) return;
    float a = 0.0f;
    for (int t = lane; t < d; t += 64) a = __builtin_fmaf(rows[(int64_t)r * d + t], rows[(int64_t)r * d + t], a);
    a = wsum(a);
    if (lane == 0) inv[r] = (a > 0.0f) ? 1.0f / __builtin_sqrtf(a) : 0.0f;
}

__global__ void fill_i32_kernel(int32_t* __restrict__ p, int64_t count, int32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// counts[l] = rows of list l; counts[nlist] = rows whose list id is out of
// range (they are left out of the index and the build fails).
__global__ void list_count_kernel(const int32_t* __restrict__ list_ids, int64_t n, int nlist,
                                  int32_t* __restrict__ counts) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t l = list_ids[i];
        atomicAdd(&counts[(l >= 0 && l < nlist) ? l : nlist], 1);
    }
}

// offsets[l] = sum of counts[0..l), offsets[nlist] = n; one block.
__global__ __launch_bounds__(1024) void list_scan_kernel(const int32_t* __restrict__ counts,
                                                         int nlist, int64_t* __restrict__ offsets) {
    __shared__ int64_t s_tot[1024];
    const int per = (nlist + 1023) / 1024;
    const int l0 = threadIdx.x * per;
    int64_t local = 0;
    for (int l = l0; l < l0 + per && l < nlist; ++l) local += counts[l];
    s_tot[threadIdx.x] = local;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t run = 0;
        for (int t = 0; t < 1024; ++t) {
            const int64_t v = s_tot[t];
            s_tot[t] = run;
            run += v;
        }
    }
    __syncthreads();
    int64_t run = s_tot[threadIdx.x];
    for (int l = l0; l < l0 + per && l < nlist; ++l) {
        offsets[l] = run;
        run += counts[l];
    }
    if (threadIdx.x == 1023) offsets[nlist] = run;
}

// Scatter of row i into its list: original id, and the key row (Flat) or
// the code row (PQ).
// Scatter of row i into its list: original id, and the key row (Flat) or
// the code row (PQ).  Codes >= ksub are counted in bad[0] (build fails).
__global__ __launch_bounds__(kIvfThreads) void list_scatter_kernel(
    const int32_t* __restrict__ list_ids, int64_t n, int nlist,
    const int64_t* __restrict__ offsets, int32_t* __restrict__ cursor,
    int32_t* __restrict__ row_ids, const uint16_t* __restrict__ keys, int64_t ld, int d,
    uint16_t* __restrict__ keys_sorted, const uint8_t* __restrict__ codes, int m, int ksub,
    uint8_t* __restrict__ codes_sorted, int32_t* __restrict__ bad) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int l = list_ids[i];
        if (l < 0 || l >= nlist) continue;
        const int64_t pos = offsets[l] + atomicAdd(&cursor[l], 1);
        row_ids[pos] = (int32_t)i;
        if (keys_sorted)
            for (int t = 0; t < d; t += 8)
                *(u32x4*)(keys_sorted + pos * d + t) = *(const u32x4*)(keys + i * ld + t);
        if (codes_sorted) {
            int nbad = 0;
            for (int j = 0; j < m; ++j) {
                const uint8_t cj = codes[i * m + j];
                nbad += cj >= ksub ? 1 : 0;
                codes_sorted[pos * m + j] = cj < ksub ? cj : 0;
            }
            if (nbad) atomicAdd(bad, nbad);
        }
    }
}

// Coarse scores: score[q][l] = sim(q, c_l) for probing; ip[q][l] = u . c_l
// with u = q (IP) or q / ||q|| (cosine), for the PQ scores.  One block per
// tile of 64 centroids and 4 * kCoarseQ queries: the tile is staged in LDS
// with coalesced loads (rows padded so that each lane's row read is free of
// bank conflicts), each lane holds one centroid in registers, each wave
// takes kCoarseQ queries, read from LDS as broadcasts (d <= KD).
constexpr int kCoarseTile = 64;
constexpr int kCoarseQ = 4;

template <int KD>
__global__ __launch_bounds__(kIvfThreads) void ivf_coarse_kernel(
    const float* __restrict__ queries, int d, int nq, const float* __restrict__ centroids,
    const float* __restrict__ cen_inv, int nlist, int cosine, float* __restrict__ score,
    float* __restrict__ ip) {
    constexpr int W = kIvfThreads / 64;
    constexpr int RS = KD + 4;                       // padded row stride (floats)
    __shared__ float4 s_c[kCoarseTile * RS / 4];
    __shared__ float4 s_q[W * kCoarseQ * KD / 4];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l0 = blockIdx.x * kCoarseTile;
    const int nt = (nlist - l0 < kCoarseTile) ? nlist - l0 : kCoarseTile;
    const int q0 = blockIdx.y * (W * kCoarseQ);
    // Tile rows l0 .. l0+nt-1 are contiguous and d % 4 == 0: float4 e of the
    // tile is centroid e / (KD/4), dims 4 (e % (KD/4)) ..; unused slots (rows
    // >= nt, dims >= d) are 0.  Every load is issued before the first store.
    constexpr int TL = kCoarseTile * KD / 4 / kIvfThreads;
    constexpr int QL = W * kCoarseQ * KD / kIvfThreads;
    float4 tv[TL];
#pragma unroll
    for (int i = 0; i < TL; ++i) {
        const int e = tid + i * kIvfThreads;
        const int r = e / (KD / 4), t = 4 * (e % (KD / 4));
        const bool in = r < nt && t < d;
        tv[i] = *(const float4*)(centroids + (int64_t)l0 * d + (in ? r * d + t : 0));
    }
    float qv[QL];
#pragma unroll
    for (int i = 0; i < QL; ++i) {
        const int e = tid + i * kIvfThreads;
        const int r = e / KD, t = e % KD;
        const bool in = q0 + r < nq && t < d;
        qv[i] = queries[in ? (int64_t)(q0 + r) * d + t : 0];
    }
#pragma unroll
    for (int i = 0; i < TL; ++i) {
        const int e = tid + i * kIvfThreads;
        const int r = e / (KD / 4), t = 4 * (e % (KD / 4));
        const bool in = r < nt && t < d;
        s_c[r * (RS / 4) + t / 4] = in ? tv[i] : float4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    float* sq = (float*)s_q;
#pragma unroll
    for (int i = 0; i < QL; ++i) {
        const int e = tid + i * kIvfThreads;
        const int r = e / KD, t = e % KD;
        sq[r * KD + t] = (q0 + r < nq && t < d) ? qv[i] : 0.0f;
    }
    __syncthreads();
    const int qw = q0 + wv * kCoarseQ;
    if (qw >= nq) return;
    float inv_q[kCoarseQ];
#pragma unroll
    for (int i = 0; i < kCoarseQ; ++i) {
        const float* qr = sq + (wv * kCoarseQ + i) * KD;
        float a = qr[lane] * qr[lane];
        if constexpr (KD > 64) a = __builtin_fmaf(qr[lane + 64], qr[lane + 64], a);
        a = wsum(a);
        inv_q[i] = (a > 0.0f) ? 1.0f / __builtin_sqrtf(a) : 0.0f;
    }
    float4 cv[KD / 4];
#pragma unroll
    for (int t = 0; t < KD / 4; ++t) cv[t] = s_c[lane * (RS / 4) + t];
    const int l = l0 + lane;
    float ci = 1.0f;
    if (cosine) ci = cen_inv[lane < nt ? l : l0];
#pragma unroll
    for (int i = 0; i < kCoarseQ; ++i) {
        const float4* qr = s_q + (wv * kCoarseQ + i) * (KD / 4);
        float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
        for (int t = 0; t < KD / 4; ++t) {
            const float4 u = qr[t];
            a0 = __builtin_fmaf(cv[t].x, u.x, a0);
            a1 = __builtin_fmaf(cv[t].y, u.y, a1);
            a0 = __builtin_fmaf(cv[t].z, u.z, a0);
            a1 = __builtin_fmaf(cv[t].w, u.w, a1);
        }
        const float dot = a0 + a1;
        if (lane < nt && qw + i < nq) {
            const int64_t o = (int64_t)(qw + i) * nlist + l;
            score[o] = cosine ? (dot * ci) * inv_q[i] : dot;
            if (ip) ip[o] = cosine ? dot * inv_q[i] : dot;
        }
    }
}

// Probe bases, per query: probe p's candidates start at the sum of the
// sizes of probes 0 .. p-1 (probe order), and the query's candidate count is
// the sum of all of them.  Every thread stores sizes into s_size and each
// probed list's first row into s_r0 (before a barrier); after it, wave 0
// writes the exclusive prefixes of the sizes into s_pre, 64 at a time, and
// returns the total (the caller's next barrier publishes s_pre).  With ip
// given, s_qc[p] = ip[list of probe p] (the PQ scores' coarse term).
__device__ __forceinline__ void load_probe_sizes(const int64_t* __restrict__ pq, int nprobe,
                                                 const int64_t* __restrict__ offsets,
                                                 int32_t* s_size, int64_t* s_r0,
                                                 const float* __restrict__ ip, float* s_qc) {
    for (int p = threadIdx.x; p < nprobe; p += kIvfThreads) {
        const int64_t l = pq[p];
        const int64_t r0 = offsets[l], r1 = offsets[l + 1];
        if (ip) s_qc[p] = ip[l];
        s_size[p] = (int32_t)(r1 - r0);
        s_r0[p] = r0;
    }
}

__device__ __forceinline__ int32_t scan_probe_sizes(const int32_t* s_size, int32_t* s_pre,
                                                    int nprobe) {
    const int lane = threadIdx.x & 63;
    int32_t carry = 0;
    for (int p0 = 0; p0 < nprobe; p0 += 64) {
        const int p = p0 + lane;
        const int32_t v = p < nprobe ? s_size[p] : 0;
        int32_t incl = v;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t t = __shfl_up(incl, off, 64);
            if (lane >= off) incl += t;
        }
        if (p < nprobe) s_pre[p] = carry + incl - v;
        carry += __shfl(incl, 63, 64);
    }
    return carry;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                                 CTRL, 0xF, 0xF, false));
}

// Sum over each aligned group of LPR lanes (the sums of an xor butterfly,
// every lane of a group with the same bits): quad xor 1, xor 2, half-row
// mirror, row mirror.
template <int LPR>
__device__ __forceinline__ float group_sum(float x) {
    static_assert(LPR == 1 || LPR == 2 || LPR == 4 || LPR == 8 || LPR == 16, "group size");
    if constexpr (LPR >= 2) x += dpp_f<0xB1>(x);
    if constexpr (LPR >= 4) x += dpp_f<0x4E>(x);
    if constexpr (LPR >= 8) x += dpp_f<0x141>(x);
    if constexpr (LPR >= 16) x += dpp_f<0x140>(x);
    return x;
}

// IVF-Flat list scan: block (p, q) scans probe p of query q; LPR lanes per
// row (16 bytes per lane, d <= 128).  Each wave takes runs of kFlatLoads
// load instructions' rows (64 / LPR rows each), and requests every key,
// norm and row id of a run together on clamped rows (rows past the list
// re-read its last row and store nothing), so a list of a few hundred rows
// is one round of loads.
constexpr int kFlatLoads = 8;

template <int KT, int LPR>
__global__ __launch_bounds__(kIvfThreads) void ivf_scan_flat_kernel(
    const uint16_t* __restrict__ keys_sorted, int d, const float* __restrict__ inv_norm,
    const int32_t* __restrict__ row_ids, const int64_t* __restrict__ offsets,
    const float* __restrict__ queries, const int64_t* __restrict__ probe, int nprobe,
    int32_t* __restrict__ count, int64_t cap, uint64_t* __restrict__ cand) {
    constexpr int RPI = 64 / LPR;                   // rows per load instruction
    constexpr int RUN = RPI * kFlatLoads;           // rows per wave and round
    __shared__ int32_t s_size[kMaxK], s_pre[kMaxK];
    __shared__ int64_t s_r0[kMaxK];
    const int q = blockIdx.y;
    const int64_t* pq = probe + (int64_t)q * nprobe;
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane / LPR, c = lane % LPR, e = c * 8;
    const bool col = e < d;
    const float* qv = queries + (int64_t)q * d;
    float qf[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const float x = qv[col ? e + t : 0];
        qf[t] = col ? x : 0.0f;
    }
    load_probe_sizes(pq, nprobe, offsets, s_size, s_r0, nullptr, nullptr);
    float qq = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) qq = __builtin_fmaf(qf[t], qf[t], qq);
    qq = group_sum<LPR>(qq);
    const float inv_q = (qq > 0.0f) ? 1.0f / __builtin_sqrtf(qq) : 0.0f;
    __syncthreads();
    if (threadIdx.x < 64) {
        const int32_t total = scan_probe_sizes(s_size, s_pre, nprobe);
        if (blockIdx.x == 0 && threadIdx.x == 0) count[q] = total;
    }
    __syncthreads();
    const int p = blockIdx.x;                       // one probe per block
    const int64_t r0 = s_r0[p], r1 = r0 + s_size[p];
    uint64_t* out = cand + (int64_t)q * cap + s_pre[p] - r0;
    // Without norms the norm load reads the query's first value (unused).
    const float* nsrc = inv_norm ? inv_norm : qv;
    const int64_t nstep = inv_norm ? 1 : 0;
    for (int64_t b0 = r0 + (int64_t)wv * RUN; b0 < r1; b0 += (int64_t)(kIvfThreads / 64) * RUN) {
        u32x4 v[kFlatLoads];
        float nv[kFlatLoads];
        int32_t rid[kFlatLoads];
#pragma unroll
        for (int u = 0; u < kFlatLoads; ++u) {
            const int64_t r = b0 + u * RPI + g;
            const int64_t rc = r < r1 ? r : r1 - 1;
            v[u] = __builtin_nontemporal_load((const u32x4*)(keys_sorted + rc * d + (col ? e : 0)));
            nv[u] = nsrc[rc * nstep];
            rid[u] = row_ids[rc];
        }
#pragma unroll
        for (int u = 0; u < kFlatLoads; ++u) {
            const u32x4 w = col ? v[u] : u32x4{0u, 0u, 0u, 0u};
            float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t x = w[k];
                float lo, hi;
                if constexpr (KT == DT_BF16) {
                    lo = __builtin_bit_cast(float, x << 16);
                    hi = __builtin_bit_cast(float, x & 0xFFFF0000u);
                } else {
                    lo = (float)__builtin_bit_cast(_Float16, (uint16_t)(x & 0xFFFFu));
                    hi = (float)__builtin_bit_cast(_Float16, (uint16_t)(x >> 16));
                }
                a0 = __builtin_fmaf(lo, qf[2 * k], a0);
                a1 = __builtin_fmaf(hi, qf[2 * k + 1], a1);
            }
            float sc = group_sum<LPR>(a0 + a1);
            if (inv_norm) sc = (sc * nv[u]) * inv_q;
            const int64_t r = b0 + u * RPI + g;
            if (c == 0 && r < r1) out[r] = pack_key(sc, (uint32_t)rid[u]);
        }
    }
}

// IVF-PQ list scan: block (g, q) builds query q's tables in LDS,
// LUT[j][c] = sum_t u[j*dsub + t] * C[j][c][t] (u = q, or q / ||q|| for
// cosine; thread c one code, its d codebook values requested up front), then
// scans probes g, g + G, ... of the query, one thread per row:
// score = u.c_l + sum_j LUT[j][code_j] (j in order).  MV = 16-byte code
// words per row (m = 16 MV): a thread's rows are pipelined, the next one
// requested before the current one is scored, and its first row before the
// barriers; MV = 0: byte loads, any m.  DS = 4: sub-vectors of 4 dims (the
// implementation details' 64 dims / 16), each code's rows requested as
// 16-byte words and each table entry one chain of 4 FMAs; DS = 0: any
// sub-vector length.
template <int MV>
struct PqCodes {
    u32x4 w[MV > 0 ? MV : 1];
    int32_t rid;
};

template <int MV>
__device__ __forceinline__ PqCodes<MV> pq_load(const uint8_t* __restrict__ codes, int m,
                                               const int32_t* __restrict__ row_ids, int64_t r) {
    PqCodes<MV> c;
#pragma unroll
    for (int v = 0; v < MV; ++v) c.w[v] = ((const u32x4*)(codes + r * m))[v];
    c.rid = row_ids[r];
    return c;
}

template <int KD, int MV, int DS>
__global__ __launch_bounds__(kIvfThreads) void ivf_scan_pq_kernel(
    const uint8_t* __restrict__ codes_sorted, int m, int ksub, const float* __restrict__ queries,
    int d, int cosine, const float* __restrict__ codebooks, const float* __restrict__ ip,
    int nlist, const int32_t* __restrict__ row_ids, const int64_t* __restrict__ offsets,
    const int64_t* __restrict__ probe, int nprobe, int32_t* __restrict__ count, int64_t cap,
    uint64_t* __restrict__ cand) {
    extern __shared__ float s_lut[];   // m * ksub
    __shared__ __attribute__((aligned(16))) float s_u[KD];
    __shared__ int32_t s_size[kMaxK], s_pre[kMaxK];
    __shared__ int64_t s_r0[kMaxK];
    __shared__ float s_qc[kMaxK];
    __shared__ float s_part[kIvfThreads / 64];
    const int q = blockIdx.y, tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int G = gridDim.x;
    const int64_t* pq = probe + (int64_t)q * nprobe;
    // First row of this thread: probe blockIdx.x, row f0 + tid (clamped to
    // a real row; rows past the list end are never scored from it).
    int p = blockIdx.x;
    const int64_t lf = pq[p];
    const int64_t f0 = offsets[lf], f1 = offsets[lf + 1];
    int64_t r = f0 + tid, r1 = f1;
    PqCodes<MV> cur{};
    if constexpr (MV > 0) {
        const int64_t rc = r < r1 ? r : (r1 > f0 ? r1 - 1 : 0);
        cur = pq_load<MV>(codes_sorted, m, row_ids, rc);
    }
    const float uq = queries[(int64_t)q * d + (tid < d ? tid : 0)];
    const int dsub = d / m;
    const int cc = tid < ksub ? tid : 0;
    constexpr int MJ = KD / 4;                      // most 4-dim sub-vectors
    float4 cb4[DS == 4 ? MJ : 1];
    float cbv[DS == 4 ? 1 : KD];
    if constexpr (DS == 4) {
        // code cc of sub-space j: C[(j * ksub + cc) * 4 .. + 4]
#pragma unroll
        for (int j = 0; j < MJ; ++j) {
            const int jj = j < m ? j : 0;
            cb4[j] = *(const float4*)(codebooks + ((int64_t)jj * ksub + cc) * 4);
        }
    } else {
        // element e = j * dsub + t of code cc lives at C[(j * ksub + cc) * dsub + t]
        int j = 0, t = 0;
#pragma unroll
        for (int e = 0; e < KD; ++e) {
            const int64_t at = ((int64_t)j * ksub + cc) * dsub + t;
            cbv[e] = codebooks[e < d ? at : 0];
            if (++t == dsub) {
                t = 0;
                ++j;
            }
        }
    }
    load_probe_sizes(pq, nprobe, offsets, s_size, s_r0, ip + (int64_t)q * nlist, s_qc);
    if (tid < KD) s_u[tid] = tid < d ? uq : 0.0f;
    const float sq = wsum(tid < d ? uq * uq : 0.0f);
    if (lane == 0) s_part[wv] = sq;
    __syncthreads();
    if (tid < 64) {
        const int32_t total = scan_probe_sizes(s_size, s_pre, nprobe);
        if (blockIdx.x == 0 && tid == 0) count[q] = total;
    }
    float qq = 0.0f;
#pragma unroll
    for (int w = 0; w < kIvfThreads / 64; ++w) qq += s_part[w];
    const float scale = cosine ? ((qq > 0.0f) ? 1.0f / __builtin_sqrtf(qq) : 0.0f) : 1.0f;
    if (tid < ksub) {
        if constexpr (DS == 4) {
#pragma unroll
            for (int j = 0; j < MJ; ++j) {
                if (j < m) {
                    const float4 u4 = *(const float4*)(s_u + 4 * j);
                    float a = __builtin_fmaf(u4.x * scale, cb4[j].x, 0.0f);
                    a = __builtin_fmaf(u4.y * scale, cb4[j].y, a);
                    a = __builtin_fmaf(u4.z * scale, cb4[j].z, a);
                    a = __builtin_fmaf(u4.w * scale, cb4[j].w, a);
                    s_lut[j * ksub + tid] = a;
                }
            }
        } else {
            int j = 0, t = 0;
            float a = 0.0f;
#pragma unroll
            for (int e = 0; e < KD; ++e) {
                if (e < d) {
                    a = __builtin_fmaf(s_u[e] * scale, cbv[e], a);
                    if (++t == dsub) {
                        s_lut[j * ksub + tid] = a;
                        a = 0.0f;
                        t = 0;
                        ++j;
                    }
                }
            }
        }
    }
    __syncthreads();
    if constexpr (MV > 0) {
        // Lanes past the end of their first list move on to their next probe.
        bool moved = false;
        while (p < nprobe && r >= r1) {
            p += G;
            if (p < nprobe) {
                r = s_r0[p] + tid;
                r1 = s_r0[p] + s_size[p];
                moved = true;
            }
        }
        if (moved && p < nprobe) cur = pq_load<MV>(codes_sorted, m, row_ids, r);
        while (p < nprobe) {
            int pn = p;
            int64_t rn = r + kIvfThreads, r1n = r1;
            while (pn < nprobe && rn >= r1n) {
                pn += G;
                if (pn < nprobe) {
                    rn = s_r0[pn] + tid;
                    r1n = s_r0[pn] + s_size[pn];
                }
            }
            const PqCodes<MV> nxt = pq_load<MV>(codes_sorted, m, row_ids, pn < nprobe ? rn : r);
            float sc = 0.0f;
#pragma unroll
            for (int j = 0; j < 16 * MV; ++j) {
                const uint32_t code = (cur.w[j / 16][(j / 4) % 4] >> (8 * (j % 4))) & 0xFFu;
                sc += s_lut[j * ksub + code];
            }
            cand[(int64_t)q * cap + s_pre[p] + (r - s_r0[p])] = pack_key(s_qc[p] + sc, (uint32_t)cur.rid);
            p = pn;
            r = rn;
            r1 = r1n;
            cur = nxt;
        }
    } else {
        for (p = blockIdx.x; p < nprobe; p += G) {
            const int64_t r0 = s_r0[p], re = r0 + s_size[p];
            uint64_t* out = cand + (int64_t)q * cap + s_pre[p] - r0;
            for (int64_t rr = r0 + tid; rr < re; rr += kIvfThreads) {
                const uint8_t* cr = codes_sorted + rr * m;
                float sc = 0.0f;
                for (int j = 0; j < m; ++j) sc += s_lut[j * ksub + cr[j]];
                out[rr] = pack_key(s_qc[p] + sc, (uint32_t)row_ids[rr]);
            }
        }
    }
}

unsigned grid_for(int64_t n, int threads) {
    int64_t b = (n + threads - 1) / threads;
    const int64_t cap = (int64_t)device_cus() * 16;
    if (b > cap) b = cap;
    return (unsigned)(b < 1 ? 1 : b);
}

}  // namespace

hipError_t launch_ivf_assign(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                             const float* centroids, int nlist, int cosine, int32_t* out_list,
                             hipStream_t stream) {
    const unsigned blocks = (unsigned)((n + kIvfThreads - 1) / kIvfThreads);
    if (d <= 64)
        hipLaunchKernelGGL(ivf_assign_kernel<64>, dim3(blocks), dim3(kIvfThreads), 0, stream,
                           (const uint16_t*)keys, key_dtype, n, d, ld, centroids, nlist, cosine,
                           out_list);
    else
        hipLaunchKernelGGL(ivf_assign_kernel<128>, dim3(blocks), dim3(kIvfThreads), 0, stream,
                           (const uint16_t*)keys, key_dtype, n, d, ld, centroids, nlist, cosine,
                           out_list);
    return hipGetLastError();
}

hipError_t launch_pq_encode(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                            const float* centroids, int nlist, const int32_t* list_ids,
                            const float* codebooks, int m, int ksub, uint8_t* codes,
                            hipStream_t stream) {
    const unsigned blocks = (unsigned)((n + kIvfThreads - 1) / kIvfThreads);
    const size_t lds = (size_t)ksub * d * sizeof(float);
    hipLaunchKernelGGL(pq_encode_kernel, dim3(blocks), dim3(kIvfThreads), lds, stream,
                       (const uint16_t*)keys, key_dtype, n, d, ld, centroids, list_ids, codebooks,
                       m, ksub, nlist, codes);
    return hipGetLastError();
}

hipError_t launch_f32_inv_norms(const float* rows, int n, int d, float* inv, hipStream_t stream) {
    hipLaunchKernelGGL(f32_inv_norm_kernel,
                       dim3((unsigned)((n + kIvfThreads / 64 - 1) / (kIvfThreads / 64))),
                       dim3(kIvfThreads), 0, stream, rows, n, d, inv);
    return hipGetLastError();
}

hipError_t launch_ivf_layout(const int32_t* list_ids, int64_t n, int nlist, const void* keys,
                             int64_t ld, int d, const uint8_t* codes, int m, int ksub,
                             int32_t* counts, int64_t* offsets, int32_t* cursor,
                             int32_t* row_ids, void* keys_sorted, uint8_t* codes_sorted,
                             hipStream_t stream) {
    // counts: nlist lists, then the out-of-range list ids, then bad codes.
    hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(nlist + 2, 256)), dim3(256), 0, stream,
                       counts, (int64_t)nlist + 2, 0);
    hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(nlist, 256)), dim3(256), 0, stream, cursor,
                       (int64_t)nlist, 0);
    hipLaunchKernelGGL(list_count_kernel, dim3(grid_for(n, 256)), dim3(256), 0, stream, list_ids,
                       n, nlist, counts);
    hipLaunchKernelGGL(list_scan_kernel, dim3(1), dim3(1024), 0, stream, counts, nlist, offsets);
    hipLaunchKernelGGL(list_scatter_kernel, dim3(grid_for(n, kIvfThreads)), dim3(kIvfThreads), 0,
                       stream, list_ids, n, nlist, offsets, cursor, row_ids,
                       (const uint16_t*)keys, ld, d, (uint16_t*)keys_sorted, codes, m, ksub,
                       codes_sorted, counts + nlist + 1);
    return hipGetLastError();
}

hipError_t launch_ivf_search(const IvfSearch& s, hipStream_t stream) {
    hipError_t e;
    constexpr int qpb = (kIvfThreads / 64) * kCoarseQ;
    const dim3 cgrid((unsigned)((s.nlist + kCoarseTile - 1) / kCoarseTile),
                     (unsigned)((s.nq + qpb - 1) / qpb));
    float* ip = s.codes_sorted ? s.coarse_ip : nullptr;
    if (s.d <= 64)
        hipLaunchKernelGGL(ivf_coarse_kernel<64>, cgrid, dim3(kIvfThreads), 0, stream, s.queries,
                           s.d, s.nq, s.centroids, s.cen_inv, s.nlist, s.cosine, s.coarse, ip);
    else
        hipLaunchKernelGGL(ivf_coarse_kernel<128>, cgrid, dim3(kIvfThreads), 0, stream, s.queries,
                           s.d, s.nq, s.centroids, s.cen_inv, s.nlist, s.cosine, s.coarse, ip);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // Probes: top-nprobe lists per query (ids only).
    if ((e = launch_topk_gather(s.coarse, s.nlist, s.nq, s.nprobe, nullptr, nullptr, 1, 1,
                                s.probe, nullptr, nullptr, nullptr, s.probe_ws, stream)) !=
        hipSuccess)
        return e;
    if (s.codes_sorted) {
        // Each block builds the query's tables once, so with many queries a
        // block takes several probes (about two blocks per compute unit).
        int g = (2 * device_cus() + s.nq - 1) / s.nq;
        g = g < 1 ? 1 : (g > s.nprobe ? s.nprobe : g);
        const dim3 grid((unsigned)g, (unsigned)s.nq);
        const size_t lds = (size_t)s.m * s.ksub * sizeof(float);
        const int mv = (s.m % 16 == 0 && s.m <= 64) ? s.m / 16 : 0;
#define SENSE_PQ_SCAN(KD, MV, DS)                                                               \
    hipLaunchKernelGGL((ivf_scan_pq_kernel<KD, MV, DS>), grid, dim3(kIvfThreads), lds, stream,   \
                       s.codes_sorted, s.m, s.ksub, s.queries, s.d, s.cosine, s.codebooks,      \
                       s.coarse_ip, s.nlist, s.row_ids, s.offsets, s.probe, s.nprobe, s.count, \
                       s.cap, s.cand)
#define SENSE_PQ_MV(KD, DS)                                                                     \
    switch (mv) {                                                                               \
        case 1: SENSE_PQ_SCAN(KD, 1, DS); break;                                                \
        case 2: SENSE_PQ_SCAN(KD, 2, DS); break;                                                \
        case 4: SENSE_PQ_SCAN(KD, 4, DS); break;                                                \
        default: SENSE_PQ_SCAN(KD, 0, DS); break;                                               \
    }
        const bool ds4 = s.d == 4 * s.m;
        if (s.d <= 64) {
            if (ds4) SENSE_PQ_MV(64, 4) else SENSE_PQ_MV(64, 0)
        } else {
            if (ds4) SENSE_PQ_MV(128, 4) else SENSE_PQ_MV(128, 0)
        }
#undef SENSE_PQ_MV
#undef SENSE_PQ_SCAN
    } else {
        const dim3 grid((unsigned)s.nprobe, (unsigned)s.nq);
        const int lanes = (s.d + 7) / 8;
        const int lpr = lanes <= 1 ? 1 : lanes <= 2 ? 2 : lanes <= 4 ? 4 : lanes <= 8 ? 8 : 16;
#define SENSE_FLAT_SCAN(KT, LPR)                                                                \
    hipLaunchKernelGGL((ivf_scan_flat_kernel<KT, LPR>), grid, dim3(kIvfThreads), 0, stream,      \
                       (const uint16_t*)s.keys_sorted, s.d, s.inv_norm, s.row_ids, s.offsets,   \
                       s.queries, s.probe, s.nprobe, s.count, s.cap, s.cand)
#define SENSE_FLAT_LPR(KT)                                                                      \
    switch (lpr) {                                                                              \
        case 1: SENSE_FLAT_SCAN(KT, 1); break;                                                  \
        case 2: SENSE_FLAT_SCAN(KT, 2); break;                                                  \
        case 4: SENSE_FLAT_SCAN(KT, 4); break;                                                  \
        case 8: SENSE_FLAT_SCAN(KT, 8); break;                                                  \
        default: SENSE_FLAT_SCAN(KT, 16); break;                                                \
    }
        if (s.key_dtype == DT_BF16) {
            SENSE_FLAT_LPR(DT_BF16)
        } else {
            SENSE_FLAT_LPR(DT_F16)
        }
#undef SENSE_FLAT_LPR
#undef SENSE_FLAT_SCAN
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_topk_keys(s.cand, s.cap, s.nq, s.k, s.spans, s.span_len, s.max_span,
                            s.span_stride, s.out_ids, s.out_scores, s.out_drafts,
                            s.out_draft_len, s.count, stream);
}

}  // namespace sense
