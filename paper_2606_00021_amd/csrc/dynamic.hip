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
    uint16_t* __restrict__ keys, int32_t* __restrict__ hist, int32_t* __restrict__ span_len) {
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
}

}  // namespace

hipError_t launch_append_rows(const void* src, int src_dtype, int key_dtype,
                              const int32_t* tokens, int d, int64_t n_old, int count,
                              int max_span, void* keys, int32_t* hist, int32_t* span_len,
                              hipStream_t stream) {
    hipLaunchKernelGGL(append_rows_kernel, dim3((unsigned)count), dim3(kAppendThreads),
                       0, stream, src, src_dtype, key_dtype, tokens, d, n_old, n_old + count,
                       max_span, (uint16_t*)keys, hist, span_len);
    return hipGetLastError();
}

}  // namespace sense
