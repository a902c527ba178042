// Single-query similarity scan for short keys (d <= 64), e.g. the 64-dim
// PCA-projected datastore of the paper's implementation details (Sec. 3.2
// Eq. 8 "sim"; Alg. 2's search step).
//
// A 64-dim bf16 row is 128 bytes, so a wave that gave every row all 64
// lanes (the long-key GEMV) would leave 7 of 8 lanes idle.  Here LPR lanes
// share a row (LPR = d/8 rounded up to a power of two, 16 bytes per lane),
// one load instruction of the wave covers 64/LPR consecutive rows (1 KiB at
// d = 64), and every lane keeps 8 loads in flight, so a wave streams 8 KiB
// per iteration.  Each row's partials are summed across its LPR lanes with
// DPP steps (quad xor 1, xor 2, then the half-row mirror: the sums of an
// xor butterfly, every lane of the group with the same bits, no LDS
// traffic), then the scores are moved so that lane L holds row base + L and
// stored 64 at a time.  Every load is unconditional on a clamped address,
// the rows' norms come with their keys, and the next iteration's loads are
// requested before the current one is scored, so a wave's loads are always
// in flight.
#include "internal.h"

namespace sense {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kSmallLoads = 8;   // loads in flight per lane per iteration

template <int KT>
__device__ __forceinline__ float dot8(const u32x4& v, const float (&q)[8]) {
    float a0 = 0.0f, a1 = 0.0f;
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
        a0 = __builtin_fmaf(lo, q[2 * w], a0);
        a1 = __builtin_fmaf(hi, q[2 * w + 1], a1);
    }
    return a0 + a1;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                                 CTRL, 0xF, 0xF, false));
}

// Sum over each aligned group of LPR lanes (LPR <= 8).
template <int LPR>
__device__ __forceinline__ float group_sum(float x) {
    static_assert(LPR == 1 || LPR == 2 || LPR == 4 || LPR == 8, "group size");
    if constexpr (LPR >= 2) x += dpp_f<0xB1>(x);    // quad_perm [1,0,3,2]
    if constexpr (LPR >= 4) x += dpp_f<0x4E>(x);    // quad_perm [2,3,0,1]
    if constexpr (LPR >= 8) x += dpp_f<0x141>(x);   // row_half_mirror
    return x;
}

// Row blocks of one iteration (512 / LPR rows) are dealt out grid-strided:
// wave w takes blocks w, w + W, w + 2W, ... (W waves in the grid), so at any
// moment the waves read neighbouring blocks (measured 7 % faster than a
// contiguous run of rows per wave).
template <int KT, int LPR>
__global__ __launch_bounds__(256) void scan_small_kernel(
    const uint16_t* __restrict__ keys, int64_t ld, int64_t n, int d,
    const float* __restrict__ query, const float* __restrict__ inv_norm,
    float* __restrict__ scores) {
    constexpr int RPI = 64 / LPR;                 // rows per load instruction
    constexpr int RPIT = kSmallLoads * RPI;       // rows per iteration
    constexpr int NG = RPIT / 64;                 // groups of 64 scores per iteration
    const int lane = threadIdx.x & 63;
    const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t r0 = wave * RPIT;
    if (r0 >= n) return;
    const int64_t r1 = n;
    const int64_t step = (int64_t)gridDim.x * 4 * RPIT;
    const int g = lane / LPR, c = lane % LPR;
    const int e = c * kLaneElems;
    const bool col = e < d;

    float q[8];
    float qq = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float x = query[col ? e + i : i];      // d % 8 == 0: in the row when col
        q[i] = col ? x : 0.0f;
        qq = __builtin_fmaf(q[i], q[i], qq);
    }
    float inv_q = 1.0f;
    if (inv_norm != nullptr) {
        const float s = group_sum<LPR>(qq);
        inv_q = (s > 0.0f) ? 1.0f / __builtin_sqrtf(s) : 0.0f;
    }

    // Keys of rows past r1 re-read row r1 - 1 (never stored); lanes past d
    // read the row's first 16 bytes and are zeroed at use.  Without norms the
    // norm load reads the query's first value (a valid address; unused).
    const float* nsrc = inv_norm ? inv_norm : query;
    const int64_t nstep = inv_norm ? 1 : 0;
    auto load_iter = [&](int64_t base, u32x4 (&b)[kSmallLoads], float (&nv)[NG]) {
#pragma unroll
        for (int u = 0; u < kSmallLoads; ++u) {
            const int64_t row = base + u * RPI + g;
            const int64_t rc = row < r1 ? row : r1 - 1;
            b[u] = __builtin_nontemporal_load((const u32x4*)(keys + rc * ld + (col ? e : 0)));
        }
#pragma unroll
        for (int k = 0; k < NG; ++k) {
            const int64_t i = base + (int64_t)k * 64 + lane;
            nv[k] = nsrc[(i < r1 ? i : r1 - 1) * nstep];
        }
    };
    // Score the rows of one iteration from its keys and norms.
    auto score_iter = [&](int64_t base, const u32x4 (&b)[kSmallLoads], const float (&nv)[NG]) {
        float p[kSmallLoads];
#pragma unroll
        for (int u = 0; u < kSmallLoads; ++u) {
            const u32x4 v = col ? b[u] : u32x4{0u, 0u, 0u, 0u};
            p[u] = group_sum<LPR>(dot8<KT>(v, q));
        }
        // Row base + u*RPI + g sits in lanes g*LPR ... ; lane L of group k
        // wants row base + 64k + L, i.e. u = k*LPR + L/RPI from lane
        // (L % RPI) * LPR.
        const int src = (lane % RPI) * LPR;
#pragma unroll
        for (int k = 0; k < NG; ++k) {
            float mine = 0.0f;
#pragma unroll
            for (int j = 0; j < LPR; ++j) {
                const float v = __shfl(p[k * LPR + j], src, 64);
                if (lane / RPI == j) mine = v;
            }
            const int64_t i = base + (int64_t)k * 64 + lane;
            if (inv_norm != nullptr) mine = (mine * nv[k]) * inv_q;
            if (i < r1) scores[i] = mine;
        }
    };
    // Two buffers taken in turn (no register copies, which would wait for
    // the loads in flight); the next iteration is requested before the
    // current one is scored.  Requests and scoring are unconditional (a
    // branch around them makes the compiler wait for every load in flight):
    // past r1 every row clamps to r1 - 1, one line per load instruction, and
    // no score is stored.
    u32x4 ka[kSmallLoads], kb[kSmallLoads];
    float na[NG], nb[NG];
    load_iter(r0, ka, na);
    for (int64_t base = r0; base < r1; base += 2 * step) {
        load_iter(base + step, kb, nb);
        score_iter(base, ka, na);
        load_iter(base + 2 * step, ka, na);
        score_iter(base + step, kb, nb);
    }
}

template <int KT, int LPR>
hipError_t launch_small_lpr(const void* keys, int64_t n, int d, int64_t ld, const float* query,
                            const float* inv_norm, float* scores, hipStream_t stream) {
    auto kern = scan_small_kernel<KT, LPR>;
    static const int per_cu = blocks_per_cu(kern, 256, 2);
    constexpr int64_t rpit = kSmallLoads * (64 / LPR);
    const int64_t max_waves = (int64_t)device_cus() * per_cu * 4;
    const int64_t row_blocks = (n + rpit - 1) / rpit;
    const int64_t waves = row_blocks < max_waves ? row_blocks : max_waves;
    const int64_t blocks = (waves + 3) / 4;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), 0, stream, (const uint16_t*)keys,
                       ld, n, d, query, inv_norm, scores);
    return hipGetLastError();
}

template <int KT>
hipError_t launch_small(const void* keys, int64_t n, int d, int64_t ld, const float* query,
                        const float* inv_norm, float* scores, hipStream_t stream) {
    const int lanes = (d + kLaneElems - 1) / kLaneElems;
    if (lanes <= 1) return launch_small_lpr<KT, 1>(keys, n, d, ld, query, inv_norm, scores, stream);
    if (lanes <= 2) return launch_small_lpr<KT, 2>(keys, n, d, ld, query, inv_norm, scores, stream);
    if (lanes <= 4) return launch_small_lpr<KT, 4>(keys, n, d, ld, query, inv_norm, scores, stream);
    return launch_small_lpr<KT, 8>(keys, n, d, ld, query, inv_norm, scores, stream);
}

}  // namespace

hipError_t launch_scan_small(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                             const float* queries, int nq, const float* inv_norm, float* scores,
                             hipStream_t stream) {
    for (int q = 0; q < nq; ++q) {
        const float* qp = queries + (int64_t)q * d;
        float* sp = scores + (int64_t)q * n;
        const hipError_t e = (key_dtype == DT_BF16)
                                 ? launch_small<DT_BF16>(keys, n, d, ld, qp, inv_norm, sp, stream)
                                 : launch_small<DT_F16>(keys, n, d, ld, qp, inv_norm, sp, stream);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace sense
