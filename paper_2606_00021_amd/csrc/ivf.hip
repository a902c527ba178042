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
//   ivf_offsets: per query, the exclusive prefix of the probed list sizes and
//     the padding of the candidate buffer;
//   ivf_lut (PQ): LUT[q][j][c] = u_j . C_j[c];
//   ivf_scan_flat / ivf_scan_pq: one block per (probe, query) scores its
//     list's rows and writes packed (score, original row) keys;
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
// with u = q (IP) or q / ||q|| (cosine), for the PQ scores.  One wave per
// centroid, the query slice in registers (d <= 128).
__global__ __launch_bounds__(kIvfThreads) void ivf_coarse_kernel(
    const float* __restrict__ queries, int d, const float* __restrict__ centroids,
    const float* __restrict__ cen_inv, int nlist, int cosine, float* __restrict__ score,
    float* __restrict__ ip) {
    const int lane = threadIdx.x & 63;
    const int q = blockIdx.y;
    const int l = blockIdx.x * (kIvfThreads / 64) + (threadIdx.x >> 6);
    const float* qv = queries + (int64_t)q * d;
    const float q0 = lane < d ? qv[lane] : 0.0f, q1 = lane + 64 < d ? qv[lane + 64] : 0.0f;
    const float qq = wsum(__builtin_fmaf(q0, q0, q1 * q1));
    const float inv_q = (qq > 0.0f) ? 1.0f / __builtin_sqrtf(qq) : 0.0f;
    if (l >= nlist) return;
    const float* c = centroids + (int64_t)l * d;
    const float c0 = lane < d ? c[lane] : 0.0f, c1 = lane + 64 < d ? c[lane + 64] : 0.0f;
    const float dot = wsum(__builtin_fmaf(q0, c0, q1 * c1));
    if (lane == 0) {
        const int64_t o = (int64_t)q * nlist + l;
        score[o] = cosine ? (dot * cen_inv[l]) * inv_q : dot;
        if (ip) ip[o] = cosine ? dot * inv_q : dot;
    }
}

// Per query: base[q][p] = sum of the sizes of probes 0..p-1 (probe lists in
// probe order), and padding keys from the total up to cap.
__global__ __launch_bounds__(kIvfThreads) void ivf_offsets_kernel(
    const int64_t* __restrict__ probe, int nprobe, const int64_t* __restrict__ offsets,
    int32_t* __restrict__ base, int32_t* __restrict__ count) {
    // Probe p's candidates start at the sum of the sizes of probes 0 .. p-1;
    // the query's candidate count is the sum of all of them.  Sizes are
    // read in parallel, then wave 0 scans them 64 at a time.
    __shared__ int32_t s_size[kMaxK];
    const int q = blockIdx.x;
    for (int p = threadIdx.x; p < nprobe; p += kIvfThreads) {
        const int64_t l = probe[(int64_t)q * nprobe + p];
        s_size[p] = (int32_t)(offsets[l + 1] - offsets[l]);
    }
    __syncthreads();
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
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
            if (p < nprobe) base[(int64_t)q * nprobe + p] = carry + incl - v;
            carry += __shfl(incl, 63, 64);
        }
        if (lane == 0) count[q] = carry;
    }
}

// LUT[q][j][c] = sum_t u[j*dsub + t] * C[j][c][t]: one block per (query,
// subspace j), thread c one code (ksub <= kIvfThreads); the thread's
// codebook entry is requested together with the query.
__global__ __launch_bounds__(kIvfThreads) void ivf_lut_kernel(
    const float* __restrict__ queries, int d, int cosine, const float* __restrict__ codebooks,
    int m, int ksub, float* __restrict__ lut) {
    __shared__ float s_u[kMaxIvfDim];
    __shared__ float s_scale;
    const int q = blockIdx.x, j = blockIdx.y;
    const int c = threadIdx.x;
    const int dsub = d / m;
    const float* cb = codebooks + ((int64_t)j * ksub + (c < ksub ? c : 0)) * dsub;
    float cbv[kMaxDsub];
#pragma unroll
    for (int t = 0; t < kMaxDsub; ++t) cbv[t] = cb[t < dsub ? t : 0];
    const float* qv = queries + (int64_t)q * d;
    for (int t = threadIdx.x; t < d; t += kIvfThreads) s_u[t] = qv[t];
    __syncthreads();
    if (threadIdx.x < 64) {
        float a = 0.0f;
        for (int t = threadIdx.x; t < d; t += 64) a = __builtin_fmaf(s_u[t], s_u[t], a);
        a = wsum(a);
        if (threadIdx.x == 0) s_scale = cosine ? ((a > 0.0f) ? 1.0f / __builtin_sqrtf(a) : 0.0f) : 1.0f;
    }
    __syncthreads();
    if (c < ksub) {
        float a = 0.0f;
#pragma unroll
        for (int t = 0; t < kMaxDsub; ++t)
            if (t < dsub) a = __builtin_fmaf(s_u[j * dsub + t] * s_scale, cbv[t], a);
        lut[((int64_t)q * m + j) * ksub + c] = a;
    }
}

// IVF-Flat list scan: one block per (probe, query); LPR lanes per row as in
// the short-key scan (d <= 128, 16 bytes per lane).
template <int KT>
__global__ __launch_bounds__(kIvfThreads) void ivf_scan_flat_kernel(
    const uint16_t* __restrict__ keys_sorted, int d, const float* __restrict__ inv_norm,
    const int32_t* __restrict__ row_ids, const int64_t* __restrict__ offsets,
    const float* __restrict__ queries, const int64_t* __restrict__ probe, int nprobe,
    const int32_t* __restrict__ base, int64_t cap, uint64_t* __restrict__ cand) {
    const int p = blockIdx.x, q = blockIdx.y;
    const int64_t l = probe[(int64_t)q * nprobe + p];
    const int64_t r0 = offsets[l], r1 = offsets[l + 1];
    const int lanes = (d + 7) / 8;
    int lpr = 1;
    while (lpr < lanes) lpr <<= 1;
    const int rpi = 64 / lpr;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int g = lane / lpr, c = lane % lpr, e = c * 8;
    const bool col = e < d;
    const float* qv = queries + (int64_t)q * d;
    float qf[8];
    float qq = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        qf[t] = col ? qv[e + t] : 0.0f;
        qq = __builtin_fmaf(qf[t], qf[t], qq);
    }
    for (int off = 1; off < lpr; off <<= 1) qq += __shfl_xor(qq, off, 64);
    const float inv_q = (qq > 0.0f) ? 1.0f / __builtin_sqrtf(qq) : 0.0f;
    uint64_t* out = cand + (int64_t)q * cap + base[(int64_t)q * nprobe + p] - r0;
    for (int64_t r = r0 + (int64_t)wv * rpi + g; r - g < r1; r += (int64_t)(kIvfThreads / 64) * rpi) {
        float a0 = 0.0f, a1 = 0.0f;
        if (col && r < r1) {
            const u32x4 v = __builtin_nontemporal_load((const u32x4*)(keys_sorted + r * d + e));
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const uint32_t u = v[w];
                float lo, hi;
                if constexpr (KT == DT_BF16) {
                    lo = __builtin_bit_cast(float, u << 16);
                    hi = __builtin_bit_cast(float, u & 0xFFFF0000u);
                } else {
                    lo = (float)__builtin_bit_cast(_Float16, (uint16_t)(u & 0xFFFFu));
                    hi = (float)__builtin_bit_cast(_Float16, (uint16_t)(u >> 16));
                }
                a0 = __builtin_fmaf(lo, qf[2 * w], a0);
                a1 = __builtin_fmaf(hi, qf[2 * w + 1], a1);
            }
        }
        float s = a0 + a1;
        for (int off = 1; off < lpr; off <<= 1) s += __shfl_xor(s, off, 64);
        if (c == 0 && r < r1) {
            if (inv_norm) s = (s * inv_norm[r]) * inv_q;
            out[r] = pack_key(s, (uint32_t)row_ids[r]);
        }
    }
}

// IVF-PQ list scan: one block per (probe, query); the query's tables in LDS,
// one thread per row: score = u.c_l + sum_j LUT[j][code_j] (j in order).
__global__ __launch_bounds__(kIvfThreads) void ivf_scan_pq_kernel(
    const uint8_t* __restrict__ codes_sorted, int m, int ksub, const float* __restrict__ lut,
    const float* __restrict__ ip, int nlist, const int32_t* __restrict__ row_ids,
    const int64_t* __restrict__ offsets, const int64_t* __restrict__ probe, int nprobe,
    const int32_t* __restrict__ base, int64_t cap, uint64_t* __restrict__ cand) {
    extern __shared__ float s_lut[];   // m * ksub
    const int p = blockIdx.x, q = blockIdx.y;
    const float* lq = lut + (int64_t)q * m * ksub;
    for (int e = threadIdx.x; e < m * ksub; e += kIvfThreads) s_lut[e] = lq[e];
    __syncthreads();
    const int64_t l = probe[(int64_t)q * nprobe + p];
    const int64_t r0 = offsets[l], r1 = offsets[l + 1];
    const float qc = ip[(int64_t)q * nlist + l];
    uint64_t* out = cand + (int64_t)q * cap + base[(int64_t)q * nprobe + p] - r0;
    for (int64_t r = r0 + threadIdx.x; r < r1; r += kIvfThreads) {
        const uint8_t* cr = codes_sorted + r * m;
        float s = 0.0f;
        for (int j = 0; j < m; ++j) s += s_lut[j * ksub + cr[j]];
        out[r] = pack_key(qc + s, (uint32_t)row_ids[r]);
    }
}

int cus() {
    static int c = 0;
    if (c == 0) {
        int dev = 0;
        hipDeviceProp_t prop;
        c = (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&prop, dev) == hipSuccess &&
             prop.multiProcessorCount > 0)
                ? prop.multiProcessorCount
                : 256;
    }
    return c;
}

unsigned grid_for(int64_t n, int threads) {
    int64_t b = (n + threads - 1) / threads;
    const int64_t cap = (int64_t)cus() * 16;
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
    hipLaunchKernelGGL(ivf_coarse_kernel,
                       dim3((unsigned)((s.nlist + kIvfThreads / 64 - 1) / (kIvfThreads / 64)),
                            (unsigned)s.nq),
                       dim3(kIvfThreads), 0, stream, s.queries, s.d, s.centroids, s.cen_inv,
                       s.nlist, s.cosine, s.coarse, s.codes_sorted ? s.coarse_ip : nullptr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // Probes: top-nprobe lists per query (ids only).
    if ((e = launch_topk_gather(s.coarse, s.nlist, s.nq, s.nprobe, nullptr, nullptr, 1, 1,
                                s.probe, nullptr, nullptr, nullptr, s.probe_ws, stream)) !=
        hipSuccess)
        return e;
    hipLaunchKernelGGL(ivf_offsets_kernel, dim3((unsigned)s.nq), dim3(kIvfThreads), 0, stream,
                       s.probe, s.nprobe, s.offsets, s.base, s.count);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const dim3 grid((unsigned)s.nprobe, (unsigned)s.nq);
    if (s.codes_sorted) {
        hipLaunchKernelGGL(ivf_lut_kernel, dim3((unsigned)s.nq, (unsigned)s.m), dim3(kIvfThreads), 0, stream,
                           s.queries, s.d, s.cosine, s.codebooks, s.m, s.ksub, s.lut);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(ivf_scan_pq_kernel, grid, dim3(kIvfThreads),
                           (size_t)s.m * s.ksub * sizeof(float), stream, s.codes_sorted, s.m,
                           s.ksub, s.lut, s.coarse_ip, s.nlist, s.row_ids, s.offsets, s.probe,
                           s.nprobe, s.base, s.cap, s.cand);
    } else if (s.key_dtype == DT_BF16) {
        hipLaunchKernelGGL(ivf_scan_flat_kernel<DT_BF16>, grid, dim3(kIvfThreads), 0, stream,
                           (const uint16_t*)s.keys_sorted, s.d, s.inv_norm, s.row_ids, s.offsets,
                           s.queries, s.probe, s.nprobe, s.base, s.cap, s.cand);
    } else {
        hipLaunchKernelGGL(ivf_scan_flat_kernel<DT_F16>, grid, dim3(kIvfThreads), 0, stream,
                           (const uint16_t*)s.keys_sorted, s.d, s.inv_norm, s.row_ids, s.offsets,
                           s.queries, s.probe, s.nprobe, s.base, s.cap, s.cand);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_topk_keys(s.cand, s.cap, s.nq, s.k, s.spans, s.span_len, s.max_span,
                            s.span_stride, s.out_ids, s.out_scores, s.out_drafts,
                            s.out_draft_len, s.final_ws, stream, s.count);
}

}  // namespace sense
