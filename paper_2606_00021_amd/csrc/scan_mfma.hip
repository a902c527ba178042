// Similarity scan for a batch of queries as a dense contraction on the
// matrix cores (Sec. 3.2 Eq. 8 "sim" for every query of a batch against
// every stored key: S = Q K^T).
//
// With Q queries each key element carries 2Q flops, so at Q >= 16 the vector
// ALUs could not keep up with HBM; v_mfma_f32_16x16x32_{bf16,f16} does.  The
// queries are the A operand (16 queries x 32 dims per instruction), the keys
// the B operand (32 dims x 16 keys); fp32 accumulation.  An fp32 query is
// split into q = hi + lo, both in the key's 16-bit type, and both halves are
// multiplied (two instructions), which keeps ~16 (bf16) / ~22 (fp16)
// mantissa bits of the query instead of 8 / 11; queries already given in the
// key type need only the hi half.
//
// Lane layout of the instruction (checked on gfx950): lane l supplies
// A[m = l%16][k = 8*(l/16) .. +8], B[k = 8*(l/16) .. +8][n = l%16] and
// receives D[m = 4*(l/16) + i][n = l%16], i = 0..3.  So each lane loads 16
// contiguous bytes of one key row straight from HBM into its B fragment: one
// load instruction covers 64 bytes of each of 16 rows.  A wave owns blocks
// of 16*T keys, holds T x MT accumulator tiles, and walks the dimension in
// steps of 32 with the next step's fragments already in flight.  Query
// fragments (at most 64 queries x d x 2 halves) are read through the caches;
// they are shared by every wave.
#include "internal.h"
#include "lds_dma.h"

namespace sense {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

template <int KT>
__device__ __forceinline__ f32x4 mfma(const u32x4& a, const u32x4& b, const f32x4& c) {
    if constexpr (KT == DT_BF16) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    } else {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    }
}

// Round-to-nearest-even fp32 -> 16-bit key type, as raw bits.
template <int KT>
__device__ __forceinline__ uint16_t to_key_bits(float x) {
    if constexpr (KT == DT_BF16) {
        const uint32_t u = __builtin_bit_cast(uint32_t, x);
        if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
        return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
    } else {
        return __builtin_bit_cast(uint16_t, (_Float16)x);
    }
}
template <int KT>
__device__ __forceinline__ float from_key_bits(uint16_t b) {
    if constexpr (KT == DT_BF16) {
        return __builtin_bit_cast(float, (uint32_t)b << 16);
    } else {
        return (float)__builtin_bit_cast(_Float16, b);
    }
}

// Pads the query batch to qpad rows and splits each fp32 value into hi + lo
// in the key type; inv_qn[q] = 1/||q|| (cosine), 1 (inner product), 0 for
// padding rows.  margin[q] is twice a bound on the difference between a
// score taken with the hi half alone on the matrix cores and the fp32
// rescore of the same row (rescore_kernel).  Cosine:
//   |A - R| <= ||q - hi|| / ||q||                      (Cauchy-Schwarz)
//            + fp32 rounding of both sums, the norms and the products
// (scores are cosines, so every term is relative to 1); inner product, with
// K the store's largest key norm (key_norm_max, NULL: margin 0):
//   |A - R| <= (||q - hi|| + rounding * ||q||) * K,
// K raised by 0.1 % for its own fp32 evaluation.  The rounding terms are
// doubled for safety and the split term raised by 1 % (its own fp32
// evaluation is good to ~d * 2^-24).  An overflowing split (an f16 hi half
// of |x| > 65504) or an infinite key gives an infinite or NaN margin: every
// row then passes.  One block (256 threads) per padded query row.
template <int KT>
__global__ __launch_bounds__(256) void query_split_kernel(const float* __restrict__ q, int nq,
                                                          int d, bool cosine,
                                                          uint16_t* __restrict__ qhi,
                                                          uint16_t* __restrict__ qlo,
                                                          float* __restrict__ inv_qn,
                                                          const float* __restrict__ key_norm_max,
                                                          float* __restrict__ margin) {
    const int row = blockIdx.x;
    float ss = 0.0f, ll = 0.0f;
    for (int t = threadIdx.x; t < d; t += 256) {
        const float x = row < nq ? q[(int64_t)row * d + t] : 0.0f;
        const uint16_t hb = to_key_bits<KT>(x);
        const float lo = x - from_key_bits<KT>(hb);
        qhi[(int64_t)row * d + t] = hb;
        qlo[(int64_t)row * d + t] = to_key_bits<KT>(lo);
        ss = __builtin_fmaf(x, x, ss);
        ll = __builtin_fmaf(lo, lo, ll);
    }
    __shared__ float s_part[2][256];
    s_part[0][threadIdx.x] = ss;
    s_part[1][threadIdx.x] = ll;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            s_part[0][threadIdx.x] += s_part[0][threadIdx.x + off];
            s_part[1][threadIdx.x] += s_part[1][threadIdx.x + off];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const float s = s_part[0][0];
        float v = 1.0f;
        if (row >= nq) v = 0.0f;
        else if (cosine) v = (s > 0.0f) ? 1.0f / __builtin_sqrtf(s) : 0.0f;
        inv_qn[row] = v;
        // summation depth of the hi-only matrix-core sum, of the rescore, and
        // of each fp32 inverse norm, plus the final products
        const float depth = (float)((d + 31) / 32 + 8) + (float)(d / 128 + 8) +
                            2.0f * (float)(d / 64 + 16) + 4.0f;
        const float rnd = depth * 5.9604645e-8f;              // x 2^-24
        const float lon = __builtin_sqrtf(s_part[1][0]);       // ||q - hi||
        float m = 0.0f;
        if (row < nq && cosine)
            m = 2.0f * (1.01f * lon * v + 2.0f * 1.01f * rnd);
        else if (row < nq && key_norm_max != nullptr)
            m = 2.0f * (1.01f * lon + 2.0f * 1.01f * rnd * __builtin_sqrtf(s)) *
                (1.001f * key_norm_max[0]);
        margin[row] = m;
    }
}

// Key-tile layout in LDS (one tile = 16 rows x 128 bytes = two 32-dimension
// steps).  Reading HBM in runs of only 64 bytes per row per load instruction
// (the matrix-core operand layout: 16 rows x 4 lanes) caps the achieved
// bandwidth near 4-5 TB/s on this device; runs of 128 bytes (8 rows per
// instruction) reach the ~7 TB/s ceiling.  So each DMA instruction fetches 8
// rows x 128 bytes and the operand layout is produced in LDS: rows 0-7 of a
// tile go to entries [0, 64), rows 8-15 to [64, 128) (16-byte entries); lane
// L = 8p + w of an instruction writes entry w of row p and fetches unit
// (w + p) mod 8 of that row, so unit u of row p sits at entry (u - p) mod 8.
// The rotation spreads the 8 rows of each half that a matrix-core read
// touches over 8 distinct 16-byte groups of a 128-byte line.  Measured with
// the LDS bank-conflict counter on this device: no conflicts with the second
// half at entry 64 (or 80), but a sixth of the read cycles in conflict with
// it at entry 72, an offset chosen for a 64-bank model in which lanes 0-15
// are served together.
constexpr int kTileVec = 128;                 // 16-byte entries per key tile
constexpr int kTileSecond = 64;               // first entry of rows 8-15

// One workgroup (4 waves) per contiguous run of key blocks; a block is 4*T
// tiles of 16 keys, T tiles per wave; MT tiles of 16 queries (nq <= 16*MT of
// them are real).  The scanned rows are rows 0, row_step, 2 row_step, ... of
// the store (a strided sample when row_step > 1).
//
// Everything the matrix cores read goes through LDS, filled by
// global_load_lds_dwordx4 (HBM/L2 -> LDS without registers) into a ring of P
// stages; a stage is two 32-dimension steps: each wave's T key tiles (private
// to the wave, laid out as above) and the 2*MT*(1+SPLIT) query fragments of
// the two steps, shared by the four waves (each wave loads its share).
// Loading stays P-1 stages ahead of the matrix cores.  Every stage a wave
// issues the same number of loads (stages past the end reload a valid
// clamped address), so the wait for a stage is a fixed vmcnt; a workgroup
// barrier then makes the other waves' query fragments visible and frees the
// slot that is refilled next.  The loop holds no register-destination global
// load, because the compiler's wait-count model does not follow LDS-DMA loads
// and would otherwise drain the whole pipeline.  Rows past n load the last
// row (their outputs are never stored); dimensions past d occur only in the
// last stage, load a clamped address and are zeroed at use.
//
// Epilogue per block (MODE): WRITE stores every score; PROJECT (the basis
// rows of a PCA projection as the queries, up to 64 of them) subtracts each
// output's centre, normalises the key's row of outputs (the four lanes
// holding it add their squares) and stores it row-major in the output type;
// FILTER keeps only
// rows whose score reaches the query's threshold (tau, the packed key of the
// k-th best row of a sample: every row of the true top k reaches it) as
// packed (score, row) keys in the query's candidate list: this wave's
// kMfmaSlots slots first (positions from ballot prefix counts), then the
// query's overflow list (atomic position).  At Q = 64 the score matrix would
// be 64 x 4 bytes per row of 16 KiB, few bytes but scattered 64-byte writes
// that cut the scan's read rate by a fifth; the survivors are ~k*row_step.
constexpr int kModeWrite = 0, kModeFilter = 1, kModeProject = 2;

template <int KT, int MT, int T, int P, bool SPLIT, int MODE>
__global__ __launch_bounds__(256) void scan_mfma_kernel(MfmaScan s, int64_t blocks_per_group) {
    constexpr bool FILTER = MODE == kModeFilter;
    constexpr int NA = MT * (SPLIT ? 2 : 1);      // query fragments per step
    constexpr int NAS = 2 * NA;                   // per stage
    constexpr int NA_W = (NAS + 3) / 4;           // loaded per wave
    constexpr int OPS = 2 * T + NA_W;             // DMA loads per wave per stage
    constexpr int KB = 64 * T;                    // keys per workgroup block
    static_assert((P - 2) * OPS < 64, "vmcnt range");
    __shared__ __attribute__((aligned(16))) u32x4 kring[P][4][T][kTileVec];
    __shared__ __attribute__((aligned(16))) u32x4 aring[P][NA_W * 4][64];
    const uint16_t* __restrict__ keys = (const uint16_t*)s.keys;
    const int d = s.d;
    const int64_t n = s.n_rows;
    const int64_t rstride = s.ld * s.row_step;    // elements between scanned rows
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int col = lane & 15, grp = lane >> 4;
    const int dp = lane >> 3;                     // DMA: row within the instruction
    const int du = ((lane & 7) + dp) & 7;         // DMA: 16-byte unit fetched
    const int64_t nblk = (n + KB - 1) / KB;
    const int64_t b0 = (int64_t)blockIdx.x * blocks_per_group;
    const int64_t b1 = (b0 + blocks_per_group < nblk) ? b0 + blocks_per_group : nblk;
    const int nks = (d + 31) / 32;
    const int nst = (nks + 1) / 2;
    const bool ragged = (d & 31) != 0;

    // This wave's share of the query fragments: fs = wv + 4*j in [0, NAS),
    // step-in-stage fs / NA, fragment fs % NA (< MT: hi tile, else lo tile).
    const uint16_t* qsrc[NA_W];
    int qstep[NA_W];
#pragma unroll
    for (int j = 0; j < NA_W; ++j) {
        int fs = wv + 4 * j;
        if (fs >= NAS) fs = NAS - 1;              // idle slot: harmless duplicate
        const int f = fs % NA;
        const uint16_t* base = (f < MT) ? s.qhi : s.qlo;
        const int mt = f % MT;
        qsrc[j] = base + (int64_t)(mt * 16 + col) * d + grp * 8;
        qstep[j] = fs / NA;
    }
    // 1/|q| of this lane's output rows, once (the batch is padded to whole
    // 16-query tiles, so every index is in bounds), and in FILTER mode their
    // threshold scores (+inf for padding queries: nothing passes; a NaN
    // threshold, from a sample of fewer than k rows, lets every row pass).
    float iq[MT][4], th[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int q = mt * 16 + grp * 4 + i;
            iq[mt][i] = s.inv_qn[q];
            if constexpr (FILTER)
                th[mt][i] = q < s.nq ? key_score((uint32_t)(s.tau[q] >> 32)) : __builtin_inff();
            if constexpr (MODE == kModeProject)   // the output's centre, mean . basis row
                th[mt][i] = (s.centre != nullptr && q < s.nq) ? s.centre[q] : 0.0f;
        }
    // FILTER: survivors so far of this wave per query (equal in a 16-lane group).
    int cnt[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) cnt[mt][i] = 0;
    const int64_t wave_slot = ((int64_t)blockIdx.x * 4 + wv) * kMfmaSlots;
    // B-operand entry of this lane inside a key tile, for unit u = 4*step + grp.
    const int ri = col >> 3, rp = col & 7;
    auto bentry = [&](int step) { return ri * kTileSecond + 8 * rp + (((4 * step + grp) - rp) & 7); };

    for (int64_t blk = b0; blk < b1; ++blk) {
        const int64_t key0 = blk * KB + (int64_t)wv * 16 * T;
        const uint16_t* kp[T][2];
        bool kv[T];
#pragma unroll
        for (int t = 0; t < T; ++t) {
            kv[t] = key0 + t * 16 + col < n;
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                int64_t row = key0 + t * 16 + 8 * i + dp;
                if (row >= n) row = n - 1;
                kp[t][i] = keys + row * rstride + du * 8;
            }
        }
        auto issue = [&](int st) {
            const int sc = st < nst ? st : nst - 1;
            const int slot = st % P;
            // kp already points at this lane's unit; past d it falls back to
            // the row's first 16 bytes (a valid address, zeroed at use).
            const int ko = (sc * 64 + du * 8 < d) ? sc * 64 : -du * 8;
#pragma unroll
            for (int t = 0; t < T; ++t)
#pragma unroll
                for (int i = 0; i < 2; ++i) dma16_nt(kp[t][i] + ko, &kring[slot][wv][t][i * kTileSecond]);
#pragma unroll
            for (int j = 0; j < NA_W; ++j) {
                const int qd = (sc * 2 + qstep[j]) * 32 + grp * 8;
                const int qo = qd < d ? qd - grp * 8 : -grp * 8;   // past d: the row's start
                dma16(qsrc[j] + qo, &aring[slot][wv + 4 * j][0]);
            }
        };
        f32x4 acc[T][MT];
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

#pragma unroll
        for (int st = 0; st < P - 1; ++st) issue(st);
        for (int st = 0; st < nst; ++st) {
            // Loads issued after stage st: stages st+1 .. st+P-2.
            wait_vmcnt<(P - 2) * OPS>();
            barrier_no_fence();
            issue(st + P - 1);                    // refills the slot read at st-1
            const int slot = st % P;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int ks = 2 * st + j;
                if (ks >= nks) break;
                const bool mask = ragged && ks == nks - 1 && ks * 32 + grp * 8 >= d;
                u32x4 a[NA];
#pragma unroll
                for (int f = 0; f < NA; ++f) {
                    a[f] = aring[slot][j * NA + f][lane];
                    if (mask) a[f] = u32x4{0u, 0u, 0u, 0u};
                }
                const int be = bentry(j);
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    u32x4 b = kring[slot][wv][t][be];
                    if (mask) b = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        acc[t][mt] = mfma<KT>(a[mt], b, acc[t][mt]);
                        if constexpr (SPLIT) acc[t][mt] = mfma<KT>(a[MT + mt], b, acc[t][mt]);
                    }
                }
            }
        }
        // Drain the surplus loads and let every wave finish reading the ring
        // before the next block's prologue refills it.
        wait_vmcnt<0>();
        barrier_no_fence();

        // Key norms of this lane's keys, all requested before any is used
        // (rows past n read the last row; their scores are not stored).
        float kscale[T];
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const int64_t key = key0 + t * 16 + col;
            kscale[t] = s.inv_norm ? s.inv_norm[(key < n ? key : n - 1) * s.row_step] : 1.0f;
        }
        // Take delivery of the scales here, once: a load still pending when
        // the conditional stores start would cost a full wait before each
        // store (pending loads and stores share one counter).
#pragma unroll
        for (int t = 0; t < T; ++t) asm volatile("" : "+v"(kscale[t]));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) asm volatile("" : "+v"(iq[mt][i]));
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const int64_t key = key0 + t * 16 + col;
            if constexpr (MODE == kModeProject) {
                // out[key][o] = (acc - centre[o]) / ||row||: the key's 16 * MT
                // outputs sit in the four lanes col, col + 16, col + 32, col + 48.
                float v[MT][4];
                float ss = 0.0f;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        v[mt][i] = acc[t][mt][i] - th[mt][i];
                        if (mt * 16 + grp * 4 + i < s.nq) ss = __builtin_fmaf(v[mt][i], v[mt][i], ss);
                    }
                ss += __shfl_xor(ss, 16, 64);
                ss += __shfl_xor(ss, 32, 64);
                float inv = 1.0f;
                if (s.normalize) inv = (ss > 0.0f) ? 1.0f / __builtin_sqrtf(ss) : 0.0f;
                if (!kv[t]) continue;
                if (s.proj_vec) {
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        const int o = mt * 16 + grp * 4;
                        if (o >= s.nq) continue;
                        const int64_t at = key * s.proj_stride + o;
                        const float y0 = v[mt][0] * inv, y1 = v[mt][1] * inv;
                        const float y2 = v[mt][2] * inv, y3 = v[mt][3] * inv;
                        if (s.proj_dtype == DT_F32) {
                            *(f32x4*)((float*)s.proj_out + at) = f32x4{y0, y1, y2, y3};
                        } else {
                            const int dt = s.proj_dtype;
                            *(u32x2*)((uint16_t*)s.proj_out + at) =
                                u32x2{(uint32_t)to_bits16(y0, dt) | ((uint32_t)to_bits16(y1, dt) << 16),
                                      (uint32_t)to_bits16(y2, dt) | ((uint32_t)to_bits16(y3, dt) << 16)};
                        }
                    }
                } else {
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const int o = mt * 16 + grp * 4 + i;
                            if (o < s.nq) {
                                const int64_t at = key * s.proj_stride + o;
                                const float y = v[mt][i] * inv;
                                if (s.proj_dtype == DT_F32) ((float*)s.proj_out)[at] = y;
                                else ((uint16_t*)s.proj_out)[at] = to_bits16(y, s.proj_dtype);
                            }
                        }
                }
            } else if constexpr (!FILTER) {
                if (!kv[t]) continue;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int q = mt * 16 + grp * 4 + i;
                        if (q < s.nq) {
                            float v = acc[t][mt][i];
                            if (s.inv_norm) v = v * kscale[t];
                            s.scores[(int64_t)q * n + key] = v * iq[mt][i];
                        }
                    }
                }
            } else {
                // One compare per score, then a branch per (query, tile) only
                // where something passed.
                float v[MT][4];
                uint64_t bal[MT][4];
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        v[mt][i] = acc[t][mt][i];
                        if (s.inv_norm) v[mt][i] = v[mt][i] * kscale[t];
                        v[mt][i] = v[mt][i] * iq[mt][i];
                        bal[mt][i] = __ballot(kv[t] & !(v[mt][i] < th[mt][i]));
                    }
                const uint32_t orig = (uint32_t)(key * s.row_step);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if (bal[mt][i] == 0) continue;
                        const int q = mt * 16 + grp * 4 + i;
                        const bool pass = (bal[mt][i] >> lane) & 1;
                        const uint32_t gm = (uint32_t)(bal[mt][i] >> (16 * grp)) & 0xFFFFu;
                        const int slot = cnt[mt][i] + __popc(gm & ((1u << col) - 1u));
                        if (pass && q < s.nq) {
                            uint64_t* cq = s.cand + (int64_t)q * s.cap;
                            const uint64_t pk = pack_key(v[mt][i], orig);
                            if (slot < kMfmaSlots) {
                                cq[wave_slot + slot] = pk;
                            } else {
                                const int pos = atomicAdd(&s.counts[q], 1);
                                cq[pos] = pk;
                            }
                        }
                        cnt[mt][i] += __popc(gm);
                    }
                }
            }
        }
    }
    if constexpr (FILTER) {
        // Unused slots become padding keys.  Lane col 0 of each group saw
        // every tile its group saw, so its counts are the group's.
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int c0 = __shfl(cnt[mt][i], lane & ~15, 64);
                const int q = mt * 16 + grp * 4 + i;
                if (q < s.nq)
                    for (int j = col; j < kMfmaSlots; j += 16)
                        if (j >= c0) s.cand[(int64_t)q * s.cap + wave_slot + j] = 0;
            }
    }
}

// Grid of the batched scan: one resident workgroup per compute unit (the
// kernels' LDS ring allows one), an equal run of blocks each.
int64_t mfma_groups(int64_t n_rows, int T) {
    const int64_t nblk = (n_rows + 64 * T - 1) / (64 * T);
    const int64_t groups_max = (int64_t)device_cus();
    int64_t bpg = (nblk + groups_max - 1) / groups_max;
    if (bpg < 1) bpg = 1;
    return (nblk + bpg - 1) / bpg;
}

template <int KT, int MT, int T, int P, bool SPLIT>
hipError_t launch_tile(const MfmaScan& s, hipStream_t stream) {
    const int64_t nblk = (s.n_rows + 64 * T - 1) / (64 * T);
    const int64_t groups = mfma_groups(s.n_rows, T);
    const int64_t bpg = (nblk + groups - 1) / groups;
    if (s.cand)
        hipLaunchKernelGGL((scan_mfma_kernel<KT, MT, T, P, SPLIT, kModeFilter>),
                           dim3((unsigned)groups), dim3(256), 0, stream, s, bpg);
    else if (s.proj_out) {
        if constexpr (SPLIT && T == 4)   // projections split the fp32 basis
            hipLaunchKernelGGL((scan_mfma_kernel<KT, MT, T, P, SPLIT, kModeProject>),
                               dim3((unsigned)groups), dim3(256), 0, stream, s, bpg);
        else
            return hipErrorInvalidValue;
    } else
        hipLaunchKernelGGL((scan_mfma_kernel<KT, MT, T, P, SPLIT, kModeWrite>),
                           dim3((unsigned)groups), dim3(256), 0, stream, s, bpg);
    return hipGetLastError();
}

// WRITE passes over few rows (a strided sample, a small store) with the hi
// half alone: blocks of 128 keys, so that every compute unit gets one (a
// block of 256 keys per unit would leave half of them idle on a 32768-row
// sample, and one unit streams a block at a fraction of the chip's rate).
template <int KT>
hipError_t launch_group_narrow(const MfmaScan& s, hipStream_t stream) {
    switch ((s.nq + 15) / 16) {
        case 1: return launch_tile<KT, 1, 2, 4, false>(s, stream);
        case 2: return launch_tile<KT, 2, 2, 4, false>(s, stream);
        case 3: return launch_tile<KT, 3, 2, 4, false>(s, stream);
        default: return launch_tile<KT, 4, 2, 4, false>(s, stream);
    }
}

template <int KT, bool SPLIT>
hipError_t launch_group(const MfmaScan& s, hipStream_t stream) {
    if constexpr (!SPLIT)
        if (s.cand == nullptr && mfma_groups(s.n_rows, 4) < (int64_t)device_cus())
            return launch_group_narrow<KT>(s, stream);
    switch ((s.nq + 15) / 16) {
        case 1: return launch_tile<KT, 1, 4, 4, SPLIT>(s, stream);
        case 2: return launch_tile<KT, 2, 4, 3, SPLIT>(s, stream);
        case 3: return launch_tile<KT, 3, 4, 3, SPLIT>(s, stream);
        default: return launch_tile<KT, 4, 4, 3, SPLIT>(s, stream);
    }
}

// Band of a hi-only filtered search: keeps, in place, the entries of query
// q's candidate list (packed (approximate score, row) keys, padding keys 0)
// whose approximate score is not below kth[q * k + k - 1] - margin[q], the
// k-th best approximate score of the list less twice the bound on
// |approximate - rescored|; a NaN on either side keeps the entry.  Every row
// whose rescored value can reach the rescored k-th best is kept.  counts[q]
// (the list's length) becomes the number kept; the order of the kept entries
// is not specified.  One block of 1024 threads per query.  Writes go only to
// positions already read: the kept count never exceeds the entries read, and
// every read of a round returns (its value decides a ballot) before the
// barrier that precedes the round's writes.
constexpr int kBandThreads = 1024;
constexpr int kBandPer = 4;
__global__ __launch_bounds__(kBandThreads) void band_kernel(uint64_t* __restrict__ cand,
                                                            int64_t cap,
                                                            const float* __restrict__ kth, int k,
                                                            const float* __restrict__ margin,
                                                            int32_t* __restrict__ counts) {
    const int q = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63;
    uint64_t* __restrict__ list = cand + (int64_t)q * cap;
    int64_t cnt = counts[q];
    cnt = cnt < 0 ? 0 : (cnt > cap ? cap : cnt);
    const float th = kth[(int64_t)q * k + (k - 1)] - margin[q];
    __shared__ int s_next;
    if (tid == 0) s_next = 0;
    __syncthreads();
    for (int64_t c0 = 0; c0 < cnt; c0 += (int64_t)kBandThreads * kBandPer) {
        uint64_t key[kBandPer];
#pragma unroll
        for (int j = 0; j < kBandPer; ++j) {
            const int64_t i = c0 + (int64_t)j * kBandThreads + tid;
            key[j] = i < cnt ? list[i] : 0ull;
        }
        uint64_t bal[kBandPer];
        int wb[kBandPer];
#pragma unroll
        for (int j = 0; j < kBandPer; ++j) {
            const bool keep = key[j] != 0ull && !(key_score((uint32_t)(key[j] >> 32)) < th);
            bal[j] = __ballot(keep);
            int b = 0;
            if (lane == 0 && bal[j]) b = atomicAdd(&s_next, __popcll(bal[j]));
            wb[j] = __shfl(b, 0, 64);
        }
        __syncthreads();
        const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
        for (int j = 0; j < kBandPer; ++j)
            if ((bal[j] >> lane) & 1ull) list[wb[j] + __popcll(bal[j] & below)] = key[j];
    }
    __syncthreads();
    if (tid == 0) counts[q] = s_next;
}

// Rescore of a band: entry e < counts[q] of query q's list (a packed key
// whose row r is what matters) becomes pack_key(R, r) with
//   R = ((sum_t q_t K[r, t]) * inv_norm[r]) * inv_qn[q]
// from the fp32 query and the stored key, as the single-query scan forms it:
// lane l takes the 16-byte units l + 64 c (c < NC = ceil(d / 512)) of the
// row, units with even c into one fp32 FMA chain and odd c into another
// (element order inside a unit), the chains are added and the wave sums its
// 64 lanes by butterfly.  One wave per entry; blocks (4 waves) stride over
// the entries of their query (blockIdx.y).  The lane's query values stay in
// registers, and a row's NC loads are all requested before the first
// product, so a row costs one round trip.
template <int KT, int NC>
__global__ __launch_bounds__(256) void rescore_kernel(uint64_t* __restrict__ cand, int64_t cap,
                                                      const int32_t* __restrict__ counts,
                                                      const uint16_t* __restrict__ keys,
                                                      int64_t ld, int d,
                                                      const float* __restrict__ queries,
                                                      const float* __restrict__ inv_norm,
                                                      const float* __restrict__ inv_qn) {
    const int q = blockIdx.y;
    const int lane = threadIdx.x & 63;
    uint64_t* __restrict__ list = cand + (int64_t)q * cap;
    int64_t cnt = counts[q];
    cnt = cnt < 0 ? 0 : (cnt > cap ? cap : cnt);
    const float* __restrict__ qrow = queries + (int64_t)q * d;
    const float iq = inv_qn[q];
    const int nu = d / 8;
    float qv[NC][8];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int u = lane + 64 * c;
        f32x4 q0 = f32x4{0.0f, 0.0f, 0.0f, 0.0f}, q1 = q0;
        if (u < nu) {
            q0 = *(const f32x4*)(qrow + u * 8);
            q1 = *(const f32x4*)(qrow + u * 8 + 4);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            qv[c][i] = q0[i];
            qv[c][4 + i] = q1[i];
        }
    }
    for (int64_t e = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); e < cnt;
         e += (int64_t)gridDim.x * 4) {
        const uint32_t r = key_row(list[e]);
        const uint16_t* __restrict__ krow = keys + (int64_t)r * ld;
        u32x4 kv[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            // a unit past the row (last chunk only) re-reads unit 0; its
            // query values are 0 and its products are skipped below
            const int u = lane + 64 * c;
            kv[c] = *(const u32x4*)(krow + (int64_t)(u < nu ? u : 0) * 8);
        }
        float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            if (c == NC - 1 && lane + 64 * c >= nu) break;
            float& a = (c & 1) ? a1 : a0;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                a = __builtin_fmaf(qv[c][i],
                                   from_key_bits<KT>((uint16_t)(kv[c][i / 2] >> (16 * (i & 1)))), a);
        }
        float a = a0 + a1;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) a += __shfl_xor(a, off, 64);
        if (lane == 0) {
            float v = a;
            if (inv_norm) v = v * inv_norm[r];
            list[e] = pack_key(v * iq, r);
        }
    }
}

template <int KT, int NC>
hipError_t launch_rescore_nc(uint64_t* cand, int64_t cap, int nq, const int32_t* counts,
                             const void* keys, int64_t ld, int d, const float* queries,
                             const float* inv_norm, const float* inv_qn, hipStream_t stream) {
    hipLaunchKernelGGL((rescore_kernel<KT, NC>), dim3(16, (unsigned)nq), dim3(256), 0, stream,
                       cand, cap, counts, (const uint16_t*)keys, ld, d, queries, inv_norm, inv_qn);
    return hipGetLastError();
}

template <int KT>
hipError_t launch_rescore_kt(uint64_t* cand, int64_t cap, int nq, const int32_t* counts,
                             const void* keys, int64_t ld, int d, const float* queries,
                             const float* inv_norm, const float* inv_qn, hipStream_t stream) {
    switch ((d + 511) / 512) {
#define SENSE_NC(N)                                                                           \
    case N:                                                                                   \
        return launch_rescore_nc<KT, N>(cand, cap, nq, counts, keys, ld, d, queries, inv_norm, \
                                        inv_qn, stream);
        SENSE_NC(1) SENSE_NC(2) SENSE_NC(3) SENSE_NC(4) SENSE_NC(5) SENSE_NC(6) SENSE_NC(7)
        SENSE_NC(8) SENSE_NC(9) SENSE_NC(10) SENSE_NC(11) SENSE_NC(12) SENSE_NC(13)
        SENSE_NC(14) SENSE_NC(15) SENSE_NC(16)
#undef SENSE_NC
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

size_t scan_mfma_scratch_bytes(int nq, int d) {
    const size_t qpad = (size_t)((nq + 15) / 16) * 16;
    const size_t half = (qpad * (size_t)d * 2 + 255) / 256 * 256;
    return 2 * half + 2 * ((qpad * 4 + 255) / 256 * 256);
}

QuerySplit query_split_parts(void* scratch, int nq, int d) {
    const int qpad = (nq + 15) / 16 * 16;
    const size_t half = ((size_t)qpad * d * 2 + 255) / 256 * 256;
    const size_t vec = ((size_t)qpad * 4 + 255) / 256 * 256;
    return QuerySplit{(uint16_t*)scratch, (uint16_t*)((char*)scratch + half),
                      (float*)((char*)scratch + 2 * half),
                      (float*)((char*)scratch + 2 * half + vec), qpad};
}

hipError_t launch_query_split(const float* queries, int nq, int d, int key_dtype, bool cosine,
                              const float* key_norm_max, void* scratch, hipStream_t stream) {
    const QuerySplit p = query_split_parts(scratch, nq, d);
    if (key_dtype == DT_BF16)
        hipLaunchKernelGGL(query_split_kernel<DT_BF16>, dim3(p.qpad), dim3(256), 0, stream,
                           queries, nq, d, cosine, p.hi, p.lo, p.inv_qn, key_norm_max, p.margin);
    else
        hipLaunchKernelGGL(query_split_kernel<DT_F16>, dim3(p.qpad), dim3(256), 0, stream,
                           queries, nq, d, cosine, p.hi, p.lo, p.inv_qn, key_norm_max, p.margin);
    return hipGetLastError();
}

int64_t mfma_scan_waves(int64_t n_rows) { return mfma_groups(n_rows, 4) * 4; }

hipError_t launch_scan_mfma_rows(const MfmaScan& s, bool split, hipStream_t stream) {
    if (s.key_dtype == DT_BF16)
        return split ? launch_group<DT_BF16, true>(s, stream) : launch_group<DT_BF16, false>(s, stream);
    return split ? launch_group<DT_F16, true>(s, stream) : launch_group<DT_F16, false>(s, stream);
}

hipError_t launch_scan_mfma(const void* keys, int key_dtype, int64_t n, int d, int64_t ld,
                            const float* queries, int nq, bool split, const float* inv_norm,
                            float* scores, void* scratch, hipStream_t stream) {
    const QuerySplit p = query_split_parts(scratch, nq, d);
    hipError_t e = launch_query_split(queries, nq, d, key_dtype, inv_norm != nullptr, nullptr,
                                      scratch, stream);
    if (e != hipSuccess) return e;
    for (int g0 = 0; g0 < nq; g0 += 64) {
        MfmaScan s{};
        s.keys = keys;
        s.key_dtype = key_dtype;
        s.ld = ld;
        s.n_rows = n;
        s.row_step = 1;
        s.d = d;
        s.qhi = p.hi + (int64_t)g0 * d;
        s.qlo = p.lo + (int64_t)g0 * d;
        s.inv_qn = p.inv_qn + g0;
        s.nq = (nq - g0 < 64) ? nq - g0 : 64;
        s.inv_norm = inv_norm;
        s.scores = scores + (int64_t)g0 * n;
        if ((e = launch_scan_mfma_rows(s, split, stream)) != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_project_mfma(const void* x, int x_dtype, int64_t n, int d_in, int64_t x_stride,
                               const float* basis, int d_out, const float* centre, int normalize,
                               void* out, int out_dtype, int64_t out_stride, void* scratch,
                               hipStream_t stream) {
    if (d_out < 1 || d_out > kMfmaProjOut) return hipErrorInvalidValue;
    const QuerySplit p = query_split_parts(scratch, d_out, d_in);
    hipError_t e = launch_query_split(basis, d_out, d_in, x_dtype, false, nullptr, scratch, stream);
    if (e != hipSuccess) return e;
    MfmaScan s{};
    s.keys = x;
    s.key_dtype = x_dtype;
    s.ld = x_stride;
    s.n_rows = n;
    s.row_step = 1;
    s.d = d_in;
    s.qhi = p.hi;
    s.qlo = p.lo;
    s.inv_qn = p.inv_qn;
    s.nq = d_out;
    s.centre = centre;
    s.proj_out = out;
    s.proj_dtype = out_dtype;
    s.proj_stride = out_stride;
    s.normalize = normalize;
    s.proj_vec = ((uintptr_t)out % 16) == 0 && out_stride % 4 == 0 && d_out % 4 == 0;
    return launch_scan_mfma_rows(s, true, stream);
}

hipError_t launch_band(uint64_t* cand, int64_t cap, int nq, const float* kth, int k,
                       const float* margin, int32_t* counts, hipStream_t stream) {
    hipLaunchKernelGGL(band_kernel, dim3((unsigned)nq), dim3(kBandThreads), 0, stream, cand, cap,
                       kth, k, margin, counts);
    return hipGetLastError();
}

hipError_t launch_rescore(uint64_t* cand, int64_t cap, int nq, const int32_t* counts,
                          const void* keys, int key_dtype, int64_t ld, int d,
                          const float* queries, const float* inv_norm, const float* inv_qn,
                          hipStream_t stream) {
    if (key_dtype == DT_BF16)
        return launch_rescore_kt<DT_BF16>(cand, cap, nq, counts, keys, ld, d, queries, inv_norm,
                                          inv_qn, stream);
    return launch_rescore_kt<DT_F16>(cand, cap, nq, counts, keys, ld, d, queries, inv_norm,
                                     inv_qn, stream);
}

}  // namespace sense
