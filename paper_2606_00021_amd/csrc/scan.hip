// Similarity scan of the SENSE retrieval step (Sec. 3.2 Eq. 8 "sim",
// Alg. 2's L2Norm and search steps), exact over all stored keys.
//
// Single-query GEMV on the vector ALUs.  The scan moves N*d*2 bytes of keys
// and does 2 flops per key element, so it is bound by HBM bandwidth; the
// kernel is laid out for that:
//   * one wave (64 lanes) owns a contiguous run of rows; for each row every
//     lane issues ceil(d/512) 16-byte loads, so one load instruction of the
//     wave reads 1 KiB of one row, fully coalesced;
//   * the next row's loads are issued before the current row is reduced
//     (two register buffers), keeping 2 rows = 16 KiB in flight per wave at
//     d = 4096;
//   * the query slice a lane needs lives in its registers for the whole run
//     (8 fp32 per 512-element chunk);
//   * per row, each lane accumulates its 8*ceil(d/512) products in fp32, then
//     the wave sums the 64 partials with DPP butterflies inside each 16-lane
//     row plus four lane reads: a fixed order, so equal rows give bit-equal
//     scores wherever they sit;
//   * scores of 64 consecutive rows are collected one per lane and written
//     with one coalesced store.
// Loads are non-temporal: every key byte is used exactly once per scan.
#include "internal.h"

namespace sense {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over the 64 lanes, same value in every lane, fixed association order.
__device__ __forceinline__ float wave_sum(float x) {
    x += dpp_f32<0xB1>(x);   // quad_perm [1,0,3,2]  (lane ^ 1)
    x += dpp_f32<0x4E>(x);   // quad_perm [2,3,0,1]  (lane ^ 2)
    x += dpp_f32<0x141>(x);  // row_half_mirror      (other quad of the 8)
    x += dpp_f32<0x140>(x);  // row_mirror           (other half of the 16)
    const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 0));
    const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 16));
    const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 32));
    const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 48));
    return (r0 + r1) + (r2 + r3);
}

template <int KT>
__device__ __forceinline__ float lo_elem(uint32_t w) {
    if constexpr (KT == DT_BF16) {
        return __builtin_bit_cast(float, w << 16);
    } else {
        return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu));
    }
}
template <int KT>
__device__ __forceinline__ float hi_elem(uint32_t w) {
    if constexpr (KT == DT_BF16) {
        return __builtin_bit_cast(float, w & 0xFFFF0000u);
    } else {
        return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
    }
}

template <int NC>
__device__ __forceinline__ void load_row(u32x4 (&buf)[NC], const uint16_t* __restrict__ row,
                                         int lane, int d) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int e = c * kWaveElems + lane * kLaneElems;
        if (c < NC - 1 || e < d) {
            buf[c] = __builtin_nontemporal_load((const u32x4*)(row + e));
        } else {
            buf[c] = u32x4{0u, 0u, 0u, 0u};
        }
    }
}

template <int KT, int NC>
__device__ __forceinline__ float lane_dot(const u32x4 (&buf)[NC], const float (&q)[NC][8]) {
    float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            a0 = __builtin_fmaf(lo_elem<KT>(buf[c][w]), q[c][2 * w], a0);
            a1 = __builtin_fmaf(hi_elem<KT>(buf[c][w]), q[c][2 * w + 1], a1);
        }
    }
    return a0 + a1;
}

// One wave per contiguous run of rows_per_wave rows.
template <int KT, int NC>
__global__ __launch_bounds__(256) void scan_gemv_kernel(
    const uint16_t* __restrict__ keys, int64_t ld, int64_t n, int d,
    const float* __restrict__ query, const float* __restrict__ inv_norm,
    float* __restrict__ scores, int64_t rows_per_wave) {
    const int lane = threadIdx.x & 63;
    const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t r0 = wave * rows_per_wave;
    if (r0 >= n) return;
    const int64_t r1 = (r0 + rows_per_wave < n) ? r0 + rows_per_wave : n;

    float q[NC][8];
    float qq = 0.0f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int e = c * kWaveElems + lane * kLaneElems;
        if (c < NC - 1 || e < d) {
            const float4 a = *(const float4*)(query + e);
            const float4 b = *(const float4*)(query + e + 4);
            q[c][0] = a.x; q[c][1] = a.y; q[c][2] = a.z; q[c][3] = a.w;
            q[c][4] = b.x; q[c][5] = b.y; q[c][6] = b.z; q[c][7] = b.w;
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) q[c][i] = 0.0f;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) qq = __builtin_fmaf(q[c][i], q[c][i], qq);
    }
    float inv_q = 1.0f;
    if (inv_norm != nullptr) {
        const float s = wave_sum(qq);
        inv_q = (s > 0.0f) ? 1.0f / __builtin_sqrtf(s) : 0.0f;
    }

    u32x4 bufa[NC], bufb[NC];
    load_row<NC>(bufa, keys + r0 * ld, lane, d);
    float mine = 0.0f;
    int64_t base = r0;  // first row of the current group of 64 scores

    auto emit = [&](int64_t r, float s) {
        const int slot = (int)(r - base);
        if (lane == slot) mine = s;
        if (slot == 63 || r == r1 - 1) {
            if (lane <= slot) {
                const int64_t i = base + lane;
                float v = mine;
                if (inv_norm != nullptr) v = (v * inv_norm[i]) * inv_q;
                scores[i] = v;
            }
            base = r + 1;
        }
    };

    for (int64_t r = r0;;) {
        if (r + 1 < r1) load_row<NC>(bufb, keys + (r + 1) * ld, lane, d);
        emit(r, wave_sum(lane_dot<KT, NC>(bufa, q)));
        if (++r >= r1) break;
        if (r + 1 < r1) load_row<NC>(bufa, keys + (r + 1) * ld, lane, d);
        emit(r, wave_sum(lane_dot<KT, NC>(bufb, q)));
        if (++r >= r1) break;
    }
}

// inv_norm[i] = 1/||row i|| (when inv_norm is not NULL) and the largest
// ||row i|| over the rows whose norm is a number, as raw bits atomically
// maxed into *max_norm_bits (when not NULL; non-negative floats order like
// their bits).  One wave per row (build-time, one pass).
template <int KT>
__global__ __launch_bounds__(256) void key_norms_kernel(const uint16_t* __restrict__ keys,
                                                        int64_t ld, int64_t n, int d,
                                                        float* __restrict__ inv_norm,
                                                        uint32_t* __restrict__ max_norm_bits) {
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * 4;
    float wmax = 0.0f;
    for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < n; r += waves) {
        float a0 = 0.0f, a1 = 0.0f;
        for (int e = lane * kLaneElems; e < d; e += kWaveElems) {
            const u32x4 v = __builtin_nontemporal_load((const u32x4*)(keys + r * ld + e));
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const float lo = lo_elem<KT>(v[w]), hi = hi_elem<KT>(v[w]);
                a0 = __builtin_fmaf(lo, lo, a0);
                a1 = __builtin_fmaf(hi, hi, a1);
            }
        }
        const float s = wave_sum(a0 + a1);
        if (inv_norm != nullptr && lane == 0)
            inv_norm[r] = (s > 0.0f) ? 1.0f / __builtin_sqrtf(s) : 0.0f;
        if (s == s) wmax = __builtin_fmaxf(wmax, __builtin_sqrtf(s));
    }
    if (max_norm_bits != nullptr && lane == 0)
        atomicMax(max_norm_bits, __builtin_bit_cast(uint32_t, wmax));
}

template <int QT>
__global__ void query_to_f32_kernel(const uint16_t* __restrict__ q, int64_t count,
                                    float* __restrict__ out) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t w = q[i];
        out[i] = (QT == DT_BF16) ? __builtin_bit_cast(float, w << 16)
                                 : (float)__builtin_bit_cast(_Float16, (uint16_t)w);
    }
}

template <int KT, int NC>
hipError_t launch_gemv_nc(const void* keys, int64_t n, int d, int64_t ld, const float* query,
                          const float* inv_norm, float* scores, hipStream_t stream) {
    auto kern = scan_gemv_kernel<KT, NC>;
    static const int per_cu = blocks_per_cu(kern, 256, 2);
    const int64_t max_blocks = (int64_t)device_cus() * per_cu;
    // Rows per wave: about 32 KiB of keys (4 rows of 4096 dims, 5 of 3584),
    // at most an equal share for a single resident wave of blocks, never
    // fewer than 2 (a small store is spread over more waves, each with its
    // next row in flight: 4096 rows of 4096 dims 21 -> 19 us).  Many rounds
    // of short-lived blocks read faster than one resident round walking
    // long row runs: 1M x 4096 in 1.20 ms against 1.26 ms, 262K x 4096 in
    // 300 us against 320 us.
    const int64_t row_bytes = 2 * (int64_t)d;
    int64_t rpw = (n + max_blocks * 4 - 1) / (max_blocks * 4);
    const int64_t by_bytes = (32768 + row_bytes - 1) / row_bytes;
    if (rpw > by_bytes) rpw = by_bytes;
    if (rpw < 2) rpw = 2;
    const int64_t waves = (n + rpw - 1) / rpw;
    const int64_t blocks = (waves + 3) / 4;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), 0, stream,
                       (const uint16_t*)keys, ld, n, d, query, inv_norm, scores, rpw);
    return hipGetLastError();
}

template <int KT>
hipError_t launch_gemv(const void* keys, int64_t n, int d, int64_t ld, const float* query,
                       const float* inv_norm, float* scores, hipStream_t stream) {
    const int nc = (d + kWaveElems - 1) / kWaveElems;
    switch (nc) {
#define SENSE_NC(N) \
    case N: return launch_gemv_nc<KT, N>(keys, n, d, ld, query, inv_norm, scores, stream);
        SENSE_NC(1) SENSE_NC(2) SENSE_NC(3) SENSE_NC(4) SENSE_NC(5) SENSE_NC(6) SENSE_NC(7)
        SENSE_NC(8) SENSE_NC(9) SENSE_NC(10) SENSE_NC(11) SENSE_NC(12) SENSE_NC(13)
        SENSE_NC(14) SENSE_NC(15) SENSE_NC(16)
#undef SENSE_NC
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

int device_cus() {
    static const int cus = [] {
        int dev = 0;
        hipDeviceProp_t prop;
        if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&prop, dev) == hipSuccess &&
            prop.multiProcessorCount > 0)
            return prop.multiProcessorCount;
        return 256;
    }();
    return cus;
}

hipError_t launch_key_norms(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                            float* inv_norm, uint32_t* max_norm_bits, hipStream_t stream) {
    int64_t blocks = (n + 3) / 4;
    const int64_t cap = (int64_t)device_cus() * 8;
    if (blocks > cap) blocks = cap;
    if (key_dtype == DT_BF16)
        hipLaunchKernelGGL(key_norms_kernel<DT_BF16>, dim3((unsigned)blocks), dim3(256), 0,
                           stream, (const uint16_t*)keys, ld, n, d, inv_norm, max_norm_bits);
    else
        hipLaunchKernelGGL(key_norms_kernel<DT_F16>, dim3((unsigned)blocks), dim3(256), 0,
                           stream, (const uint16_t*)keys, ld, n, d, inv_norm, max_norm_bits);
    return hipGetLastError();
}

hipError_t launch_query_to_f32(const void* q, int q_dtype, int nq, int d, float* out,
                               hipStream_t stream) {
    const int64_t count = (int64_t)nq * d;
    if (q_dtype == DT_F32)
        return hipMemcpyAsync(out, q, count * sizeof(float), hipMemcpyDeviceToDevice, stream);
    int64_t blocks = (count + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    if (q_dtype == DT_BF16)
        hipLaunchKernelGGL(query_to_f32_kernel<DT_BF16>, dim3((unsigned)blocks), dim3(256), 0,
                           stream, (const uint16_t*)q, count, out);
    else
        hipLaunchKernelGGL(query_to_f32_kernel<DT_F16>, dim3((unsigned)blocks), dim3(256), 0,
                           stream, (const uint16_t*)q, count, out);
    return hipGetLastError();
}

hipError_t launch_scan(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                       const float* queries, int nq, bool split, const float* inv_norm,
                       float* scores, void* scratch, hipStream_t stream) {
    if (nq >= kMfmaMinQueries)
        return launch_scan_mfma(keys, key_dtype, n, d, ld, queries, nq, split, inv_norm, scores,
                                scratch, stream);
    for (int q = 0; q < nq; ++q) {
        const float* qp = queries + (int64_t)q * d;
        float* sp = scores + (int64_t)q * n;
        const hipError_t e =
            (key_dtype == DT_BF16)
                ? launch_gemv<DT_BF16>(keys, n, d, ld, qp, inv_norm, sp, stream)
                : launch_gemv<DT_F16>(keys, n, d, ld, qp, inv_norm, sp, stream);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace sense
