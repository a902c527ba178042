// PCA projection with L2 normalisation: Alg. 2's query k = L2Norm(PCA(h))
// and the datastore projection Z of Sec. 3.2 Eq. 6 (the implementation
// details project 4096-dim hidden states to 64 dims and L2-normalise them).
//
//   out[i][o] = sum_t (x[i][t] - mean[t]) * basis[o][t],  then row i / ||row i||
//
// Two routes:
//   * many 16-bit rows (building a projected datastore) is a dense
//     contraction N x d_in x d_out: it runs on the matrix cores through the
//     batched similarity kernel with the basis rows as the "queries" (fp32
//     basis split into hi + lo halves of the key type).  Up to 64 outputs
//     its epilogue subtracts mean . w_o, normalises each row and stores it
//     in the output type; beyond that it writes S[o][i] = x_i . w_o and
//     project_finish does the same from S;
//   * a few rows (queries) or fp32 / unaligned rows: blocks of 2 rows x 16
//     outputs centre their rows in LDS and form the dot products (one wave
//     per output, fixed-order sums); then one wave per row normalises and
//     stores it.
#include "internal.h"

namespace sense {
namespace {

constexpr int kProjThreads = 256;

// Sum over the 64 lanes by an xor butterfly: every lane ends with the same
// bits (each step adds the same two operands in every lane pair).
__device__ __forceinline__ float wsum(float x) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) x += __shfl_xor(x, off, 64);
    return x;
}

__device__ __forceinline__ void store_out(void* p, int dt, int64_t i, float v) {
    if (dt == DT_F32) ((float*)p)[i] = v;
    else ((uint16_t*)p)[i] = to_bits16(v, dt);
}

// centre[o] = mean . basis[o]  (one wave per output).
__global__ __launch_bounds__(kProjThreads) void project_center_kernel(
    const float* __restrict__ mean, const float* __restrict__ basis, int d_in, int d_out,
    float* __restrict__ centre) {
    const int lane = threadIdx.x & 63;
    const int o = blockIdx.x * (kProjThreads / 64) + (threadIdx.x >> 6);
    if (o >= d_out) return;
    float a = 0.0f;
    for (int t = lane; t < d_in; t += 64) a = __builtin_fmaf(mean[t], basis[(int64_t)o * d_in + t], a);
    a = wsum(a);
    if (lane == 0) centre[o] = a;
}

// Rows [i0, i0 + kFinRows) of S (d_out x n): subtract the centre, normalise,
// store row-major in the output type.
constexpr int kFinRows = 32;

__global__ __launch_bounds__(kProjThreads) void project_finish_kernel(
    const float* __restrict__ s, int64_t n, int d_out, const float* __restrict__ centre,
    int normalize, void* __restrict__ out, int out_dtype, int64_t out_stride) {
    __shared__ float tile[kFinRows * (kMaxProjOut + 1)];
    const int ld = d_out + 1;
    const int64_t i0 = (int64_t)blockIdx.x * kFinRows;
    for (int idx = threadIdx.x; idx < kFinRows * d_out; idx += kProjThreads) {
        const int o = idx / kFinRows, r = idx - o * kFinRows;
        const int64_t i = i0 + r;
        float v = 0.0f;
        if (i < n) v = s[(int64_t)o * n + i] - (centre ? centre[o] : 0.0f);
        tile[r * ld + o] = v;
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    for (int r = wv; r < kFinRows; r += kProjThreads / 64) {
        const int64_t i = i0 + r;
        if (i >= n) break;                               // uniform over the wave
        float inv = 1.0f;
        if (normalize) {
            float ss = 0.0f;
            for (int o = lane; o < d_out; o += 64) ss = __builtin_fmaf(tile[r * ld + o], tile[r * ld + o], ss);
            ss = wsum(ss);
            inv = (ss > 0.0f) ? 1.0f / __builtin_sqrtf(ss) : 0.0f;
        }
        for (int o = lane; o < d_out; o += 64)
            store_out(out, out_dtype, i * out_stride + o, tile[r * ld + o] * inv);
    }
}

// Direct route, step 1: raw[i][o] = (x_i - mean) . w_o by tiles of kTileRows
// rows x kTileOuts outputs, one block of 1024 threads (one wave per output)
// per tile, so that the basis is read by many CUs at once while each block
// reads its rows once.  The centred rows go to LDS (each thread's loads
// issued together, on clamped indices); each wave then streams its basis row
// (16-byte loads when the basis is 16-byte aligned, else one float per lane)
// against them in batches of loads issued together, and a fixed-order
// butterfly sums the lanes.
constexpr int kTileThreads = 1024;
constexpr int kTileOuts = kTileThreads / 64;
constexpr int kTileRows = 2;

template <int XT>
__device__ __forceinline__ float load_xt(const void* p, int64_t i) {
    if constexpr (XT == DT_F32) return ((const float*)p)[i];
    const uint16_t b = ((const uint16_t*)p)[i];
    if constexpr (XT == DT_F16) return (float)__builtin_bit_cast(_Float16, b);
    return __builtin_bit_cast(float, (uint32_t)b << 16);
}

template <int XT, bool VEC>
__global__ __launch_bounds__(kTileThreads) void project_tile_kernel(
    const void* __restrict__ x, int64_t x_stride, int64_t n, int d_in,
    const float* __restrict__ mean, const float* __restrict__ basis, int d_out,
    float* __restrict__ raw) {
    __shared__ __attribute__((aligned(16))) float s_c[kTileRows][kMaxDim];
    const int64_t i0 = (int64_t)blockIdx.x * kTileRows;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;

    constexpr int kA = kMaxDim / kTileThreads;
    const float* m = mean ? mean : basis;          // a valid address; unused without a mean
#pragma unroll
    for (int r = 0; r < kTileRows; ++r) {
        const int64_t i = (i0 + r < n) ? i0 + r : n - 1;
        float xv[kA], mv[kA];
#pragma unroll
        for (int e = 0; e < kA; ++e) {
            const int t = tid + e * kTileThreads;
            const int tc = t < d_in ? t : d_in - 1;
            xv[e] = load_xt<XT>(x, i * x_stride + tc);
            mv[e] = m[tc];
        }
#pragma unroll
        for (int e = 0; e < kA; ++e) {
            const int t = tid + e * kTileThreads;
            if (t < d_in) s_c[r][t] = xv[e] - (mean ? mv[e] : 0.0f);
        }
    }
    __syncthreads();

    const int o = blockIdx.y * kTileOuts + wv;
    if (o >= d_out) return;                          // uniform over the wave
    const float* w = basis + (int64_t)o * d_in;
    float a[kTileRows];
#pragma unroll
    for (int r = 0; r < kTileRows; ++r) a[r] = 0.0f;
    if constexpr (VEC) {
        constexpr int kB = 16;                      // 16-byte loads per batch
        for (int j0 = 0; 256 * j0 < d_in; j0 += kB) {
            float4 wq[kB];
#pragma unroll
            for (int u = 0; u < kB; ++u) {
                const int t = 4 * lane + 256 * (j0 + u);
                wq[u] = *(const float4*)(w + (t < d_in ? t : 0));
            }
#pragma unroll
            for (int u = 0; u < kB; ++u) {
                const int t = 4 * lane + 256 * (j0 + u);
                if (t < d_in) {
#pragma unroll
                    for (int r = 0; r < kTileRows; ++r) {
                        const float4 c = *(const float4*)(&s_c[r][t]);
                        a[r] = __builtin_fmaf(c.x, wq[u].x, a[r]);
                        a[r] = __builtin_fmaf(c.y, wq[u].y, a[r]);
                        a[r] = __builtin_fmaf(c.z, wq[u].z, a[r]);
                        a[r] = __builtin_fmaf(c.w, wq[u].w, a[r]);
                    }
                }
            }
        }
    } else {
        constexpr int kB = 32;                      // scalar loads per batch
        for (int j0 = 0; 64 * j0 < d_in; j0 += kB) {
            float wq[kB];
#pragma unroll
            for (int u = 0; u < kB; ++u) {
                const int t = lane + 64 * (j0 + u);
                wq[u] = w[t < d_in ? t : 0];
            }
#pragma unroll
            for (int u = 0; u < kB; ++u) {
                const int t = lane + 64 * (j0 + u);
                if (t < d_in) {
#pragma unroll
                    for (int r = 0; r < kTileRows; ++r) a[r] = __builtin_fmaf(s_c[r][t], wq[u], a[r]);
                }
            }
        }
    }
#pragma unroll
    for (int r = 0; r < kTileRows; ++r) {
        const float v = wsum(a[r]);
        if (lane == 0 && i0 + r < n) raw[(i0 + r) * d_out + o] = v;
    }
}

// Direct route, step 2: normalise row i and store it in the output type.
__global__ __launch_bounds__(64) void project_norm_kernel(
    const float* __restrict__ raw, int d_out, int normalize, void* __restrict__ out,
    int out_dtype, int64_t out_stride) {
    const int64_t i = blockIdx.x;
    const int lane = threadIdx.x;
    const float* r = raw + i * d_out;
    float v[kMaxProjOut / 64];
#pragma unroll
    for (int e = 0; e < kMaxProjOut / 64; ++e) {
        const int o = lane + 64 * e;
        v[e] = r[o < d_out ? o : 0];
    }
    float inv = 1.0f;
    if (normalize) {
        float ss = 0.0f;
#pragma unroll
        for (int e = 0; e < kMaxProjOut / 64; ++e)
            if (lane + 64 * e < d_out) ss = __builtin_fmaf(v[e], v[e], ss);
        ss = wsum(ss);
        inv = (ss > 0.0f) ? 1.0f / __builtin_sqrtf(ss) : 0.0f;
    }
#pragma unroll
    for (int e = 0; e < kMaxProjOut / 64; ++e) {
        const int o = lane + 64 * e;
        if (o < d_out) store_out(out, out_dtype, i * out_stride + o, v[e] * inv);
    }
}

template <int XT>
void launch_tiles(const void* x, int64_t n, int d_in, int64_t x_stride, const float* mean,
                  const float* basis, int d_out, float* raw, hipStream_t stream) {
    const dim3 grid((unsigned)((n + kTileRows - 1) / kTileRows),
                    (unsigned)((d_out + kTileOuts - 1) / kTileOuts));
    if (((uintptr_t)basis % 16) == 0)
        hipLaunchKernelGGL((project_tile_kernel<XT, true>), grid, dim3(kTileThreads), 0, stream,
                           x, x_stride, n, d_in, mean, basis, d_out, raw);
    else
        hipLaunchKernelGGL((project_tile_kernel<XT, false>), grid, dim3(kTileThreads), 0, stream,
                           x, x_stride, n, d_in, mean, basis, d_out, raw);
}

}  // namespace

bool project_uses_mfma(int x_dtype, const void* x, int64_t x_stride, int64_t n) {
    return x_dtype != DT_F32 && n >= kProjMfmaMinRows && ((uintptr_t)x % 16) == 0 &&
           x_stride % 8 == 0;
}

// Workspace: [centre (d_out fp32) | S (d_out x n fp32; not for a fused
// projection) | MFMA scratch].
static size_t up256(size_t x) { return (x + 255) / 256 * 256; }

static bool project_fused(int d_out) { return d_out <= kMfmaProjOut; }

size_t project_workspace_bytes(int x_dtype, int64_t n, int d_in, int d_out) {
    if (n == 0) return 0;
    const bool mfma = x_dtype != DT_F32 && n >= kProjMfmaMinRows;
    size_t bytes = up256((size_t)d_out * sizeof(float));
    if (!(mfma && project_fused(d_out))) bytes += up256((size_t)d_out * n * sizeof(float));
    if (mfma) bytes += up256(scan_mfma_scratch_bytes(d_out, d_in));
    return bytes;
}

hipError_t launch_project(const void* x, int x_dtype, int64_t n, int d_in, int64_t x_stride,
                          const float* mean, const float* basis, int d_out, int normalize,
                          void* out, int out_dtype, int64_t out_stride, void* workspace,
                          hipStream_t stream) {
    if (n == 0) return hipSuccess;
    char* ws = (char*)workspace;
    const size_t c_bytes = up256((size_t)d_out * sizeof(float));
    float* centre = mean ? (float*)ws : nullptr;
    float* s = (float*)(ws + c_bytes);
    hipError_t e;
    if (!project_uses_mfma(x_dtype, x, x_stride, n)) {
        if (x_dtype == DT_F32)
            launch_tiles<DT_F32>(x, n, d_in, x_stride, mean, basis, d_out, s, stream);
        else if (x_dtype == DT_F16)
            launch_tiles<DT_F16>(x, n, d_in, x_stride, mean, basis, d_out, s, stream);
        else
            launch_tiles<DT_BF16>(x, n, d_in, x_stride, mean, basis, d_out, s, stream);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(project_norm_kernel, dim3((unsigned)n), dim3(64), 0, stream, s, d_out,
                           normalize, out, out_dtype, out_stride);
        return hipGetLastError();
    }
    if (mean) {
        hipLaunchKernelGGL(project_center_kernel,
                           dim3((unsigned)((d_out + kProjThreads / 64 - 1) / (kProjThreads / 64))),
                           dim3(kProjThreads), 0, stream, mean, basis, d_in, d_out, centre);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (project_fused(d_out))
        return launch_project_mfma(x, x_dtype, n, d_in, x_stride, basis, d_out, centre, normalize,
                                   out, out_dtype, out_stride, ws + c_bytes, stream);
    void* scratch = ws + c_bytes + up256((size_t)d_out * n * sizeof(float));
    if ((e = launch_scan_mfma(x, x_dtype, n, d_in, x_stride, basis, d_out, true, nullptr, s,
                              scratch, stream)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(project_finish_kernel, dim3((unsigned)((n + kFinRows - 1) / kFinRows)),
                       dim3(kProjThreads), 0, stream, s, n, d_out, centre, normalize, out,
                       out_dtype, out_stride);
    return hipGetLastError();
}

}  // namespace sense
