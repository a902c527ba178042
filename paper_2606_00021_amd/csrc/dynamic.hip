// Append step of the dynamic context cache C_d (Alg. 1's retriever update;
// Alg. 2's dynamic search reads the cache like any other index).
//
// The cache stores, for every generated position p, the key that predicted
// token p and the token itself.  The continuation of row p is the generated
// text from p on: tokens[p .. p + M), cut at the end of the history.  The
// tokens are kept as one array, so the continuation table is that array read
// with a row stride of one token; only the lengths min(M, n - p) of the last
// M - 1 old rows change when rows are appended.
#include "internal.h"

namespace sense {
namespace {

constexpr int kAppendThreads = 256;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int CTRL>
__device__ __forceinline__ float dpp_move(float x) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over the 64 lanes in the association order the index build uses for
// key norms (pairs, quads, halves of 8 and 16, then the four rows), so that
// both give the same bits.
__device__ __forceinline__ float norm_wave_sum(float x) {
    x += dpp_move<0xB1>(x);
    x += dpp_move<0x4E>(x);
    x += dpp_move<0x141>(x);
    x += dpp_move<0x140>(x);
    const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 0));
    const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 16));
    const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 32));
    const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 48));
    return (r0 + r1) + (r2 + r3);
}

// The low and high element of a word of two stored key values, exactly.
__device__ __forceinline__ float low_value(uint32_t w, int key_dtype) {
    return key_dtype == DT_BF16 ? __builtin_bit_cast(float, w << 16)
                                : (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu));
}
__device__ __forceinline__ float high_value(uint32_t w, int key_dtype) {
    return key_dtype == DT_BF16 ? __builtin_bit_cast(float, w & 0xFFFF0000u)
                                : (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
}

__device__ inline float load_as_float(const void* p, int dt, int64_t i) {
    if (dt == DT_F32) return ((const float*)p)[i];
    const uint16_t b = ((const uint16_t*)p)[i];
    if (dt == DT_F16) {
        _Float16 h;
        __builtin_memcpy(&h, &b, 2);
        return (float)h;
    }
    const uint32_t u = (uint32_t)b << 16;
    float f;
    __builtin_memcpy(&f, &u, 4);
    return f;
}

// Block b appends row n_old + b: its key (converted to the key type) and
// token.  Block 0 also refreshes the lengths of the M - 1 rows before n_old.
__global__ __launch_bounds__(kAppendThreads) void append_rows_kernel(
    const void* __restrict__ src, int src_dtype, int key_dtype,
    const int32_t* __restrict__ tokens, int d, int64_t n_old, int64_t n_new, int max_span,
    uint16_t* __restrict__ keys, int32_t* __restrict__ hist, int32_t* __restrict__ span_len,
    float* __restrict__ inv_norm, uint32_t* __restrict__ max_norm_bits) {
    const int64_t b = blockIdx.x;
    const int64_t row = n_old + b;
    uint16_t* dst = keys + row * d;
    for (int t = threadIdx.x; t < d; t += kAppendThreads)
        dst[t] = to_bits16(load_as_float(src, src_dtype, b * d + t), key_dtype);
    if (threadIdx.x == 0) {
        hist[row] = tokens[b];
        const int64_t left = n_new - row;
        span_len[row] = (int32_t)(left < max_span ? left : max_span);
    }
    if (b == 0) {
        const int64_t lo = n_old - (max_span - 1) > 0 ? n_old - (max_span - 1) : 0;
        for (int64_t r = lo + threadIdx.x; r < n_old; r += kAppendThreads) {
            const int64_t left = n_new - r;
            span_len[r] = (int32_t)(left < max_span ? left : max_span);
        }
    }
    if (inv_norm != nullptr || max_norm_bits != nullptr) {   // uniform over the grid
        // 1/||k|| of the stored row, summed exactly as the index build sums
        // it (lane l takes 8 elements in every 512, even and odd elements in
        // two chains, then the wave sum), so an appended row's value is
        // bit-identical to a rebuilt index's.
        __syncthreads();                            // the block's row stores are visible
        if (threadIdx.x < 64) {
            const int lane = threadIdx.x;
            float a0 = 0.0f, a1 = 0.0f;
            for (int e = lane * kLaneElems; e < d; e += kWaveElems) {
                const u32x4 v = *(const u32x4*)(dst + e);
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const float lo = low_value(v[w], key_dtype);
                    const float hi = high_value(v[w], key_dtype);
                    a0 = __builtin_fmaf(lo, lo, a0);
                    a1 = __builtin_fmaf(hi, hi, a1);
                }
            }
            const float s = norm_wave_sum(a0 + a1);
            if (inv_norm != nullptr && lane == 0)
                inv_norm[row] = (s > 0.0f) ? 1.0f / __builtin_sqrtf(s) : 0.0f;
            // inner product: the cache's largest key norm (rows whose norm is
            // a number), as the index build keeps it
            if (max_norm_bits != nullptr && lane == 0 && s == s)
                atomicMax(max_norm_bits, __builtin_bit_cast(uint32_t, __builtin_sqrtf(s)));
        }
    }
}

}  // namespace

hipError_t launch_append_rows(const void* src, int src_dtype, int key_dtype,
                              const int32_t* tokens, int d, int64_t n_old, int count,
                              int max_span, void* keys, int32_t* hist, int32_t* span_len,
                              float* inv_norm, uint32_t* max_norm_bits, hipStream_t stream) {
    hipLaunchKernelGGL(append_rows_kernel, dim3((unsigned)count), dim3(kAppendThreads),
                       0, stream, src, src_dtype, key_dtype, tokens, d, n_old, n_old + count,
                       max_span, (uint16_t*)keys, hist, span_len, inv_norm, max_norm_bits);
    return hipGetLastError();
}

}  // namespace sense
