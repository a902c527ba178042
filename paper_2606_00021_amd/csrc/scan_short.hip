// Batched similarity scan of short keys (d <= 64, e.g. the 64-dim PCA keys)
// on the matrix cores, with an optional filter that keeps only rows able to
// enter a query's top k (Sec. 3.2 Eq. 8 for a batch of queries; the top-N'
// retrieval of Eq. 7).
//
// A 64-dim key is 128 bytes, so the long-key MFMA design (a ring of key
// stages walking d) has nothing to pipeline across.  Here every wave keeps
// the whole query batch (up to 64 queries x 64 dims, hi and lo halves) in
// registers as A fragments and streams 16-key tiles as B fragments straight
// from HBM: lane l loads 16 bytes of key (base + l%16) at dims 8*(l/16) and
// 32 + 8*(l/16), so one tile is 16 contiguous rows (2 KiB at d = 64).  Four
// tiles are in flight per wave.  Per tile: 4 query tiles x 2 k-steps x
// (hi, lo) MFMA 16x16x32 instructions.
//
// The 64 x n score matrix would be 256 MB at n = 1M: writing it and reading
// it back for the top-k costs more than reading the keys.  So the scan runs
// twice: first over a strided sample of rows writing scores, whose per-query
// k-th best packed key tau bounds the final k-th best from below; then over
// all rows, keeping only rows whose packed key reaches tau: each wave has a
// few slots per query (about k * rows_per_wave / sample rows survive per
// wave, ~1-2 at the bench shape), filled in order (ballot + popcount), and a
// query's overflow list takes what does not fit.
// Every true top-k row passes, so the result is exact; the scores of both
// passes come from the same instructions, hence the same bits.
#include "internal.h"
#include "lds_dma.h"

namespace sense {

int64_t short_rows_per_wave(int64_t n_rows);

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

constexpr int kShortThreads = 256;
constexpr int kShortDepth = 4;     // 16-key tiles in flight per wave
static_assert(kShortSlots <= 16, "one padding slot per lane of a 16-lane group");

template <int KT>
__device__ __forceinline__ f32x4 mfma(const u32x4& a, const u32x4& b, const f32x4& c) {
    if constexpr (KT == DT_BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// NT query tiles of 16, KS k-steps of 32 dims (d <= 32 * KS).
template <int KT, int NT, int KS, bool SPLIT, bool FILTER>
__global__ __launch_bounds__(kShortThreads, 2) void scan_short_kernel(ShortScan s,
                                                                  int64_t rows_per_wave) {
    // Per query: {scale 1/|q|, threshold score}, in LDS (read in the
    // epilogue without a wait on the key loads in flight, and without
    // registers).  A row passes the filter when its score is not below the
    // threshold score: a superset of the rows whose packed key reaches tau
    // (a NaN threshold, from a NaN tau or a sample without k rows, lets
    // every row through).  Queries past nq get +inf and are also checked by
    // index before anything is stored.
    __shared__ float2 s_qt[64];
    if (threadIdx.x < 64) {
        const int q = threadIdx.x;
        float th = 0.0f;
        if constexpr (FILTER)
            th = q < s.nq ? key_score((uint32_t)(s.tau[q] >> 32)) : __builtin_inff();
        s_qt[q] = float2{q < 16 * NT ? s.inv_qn[q] : 0.0f, th};
    }
    __syncthreads();
    const int lane = threadIdx.x & 63;
    // The wave index is uniform: the row loop below is then a scalar loop.
    const int64_t wave = (int64_t)blockIdx.x * (kShortThreads / 64) +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t r0 = wave * rows_per_wave;
    if (r0 >= s.n_rows) return;                      // uniform over the wave
    const int64_t r1 = (r0 + rows_per_wave < s.n_rows) ? r0 + rows_per_wave : s.n_rows;
    const int col = lane & 15, grp = lane >> 4;

    // Query fragments: A[m = col][k = 8*grp + 32*ks], for every query tile.
    u32x4 ahi[NT][KS], alo[NT][KS];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int dim = 8 * grp + 32 * ks;
            const int64_t qrow = 16 * t + col;
            const bool ok = dim < s.d;
            ahi[t][ks] = ok ? *(const u32x4*)(s.qhi + qrow * s.d + dim) : u32x4{0u, 0u, 0u, 0u};
            if constexpr (SPLIT)
                alo[t][ks] = ok ? *(const u32x4*)(s.qlo + qrow * s.d + dim) : u32x4{0u, 0u, 0u, 0u};
        }
    }
    int cnt[NT][4];       // FILTER: survivors so far per query (same in a 16-lane group)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) cnt[t][i] = 0;

    // This lane's key row advances by 16 rows per tile: pointers step by a
    // fixed stride (no 64-bit multiplies per tile).  Every load is issued
    // unconditionally, so the compiler can count the loads in flight exactly
    // (a load under a branch makes it wait for all of them): rows past r1
    // re-read the lane's last row (their scores are discarded), dims past d
    // read dim 0 and are zeroed before use.  Everything an iteration reads
    // comes in with the tile (keys and the key norm): a load issued later and
    // consumed earlier would make the wave wait for all the tiles in flight
    // before it.
    const int64_t key_step = 16 * s.row_step * s.ld;
    const int64_t norm_step = s.inv_norm ? 16 * s.row_step : 0;
    const int64_t row_first = (r0 + col < r1) ? r0 + col : r1 - 1;
    const uint16_t* kp = (const uint16_t*)s.keys + row_first * s.row_step * s.ld;
    // Without key norms the norm load reads a fixed valid word (unused).
    const float* np = s.inv_norm ? s.inv_norm + row_first * s.row_step : s.inv_qn;
    const bool dim0 = 8 * grp < s.d;                 // this lane's dims hold key elements
    const bool dim1 = 8 * grp + 32 < s.d;            // ... in the second k-step
    const int off0 = dim0 ? 8 * grp : 0;
    const int off1 = dim1 ? 8 * grp + 32 : 0;
    int64_t lr = r0 + col;                           // row of the next tile to load
    auto load_tile = [&](u32x4 (&b)[KS], float& kn) {
        b[0] = __builtin_nontemporal_load((const u32x4*)(kp + off0));
        if constexpr (KS == 2) b[1] = __builtin_nontemporal_load((const u32x4*)(kp + off1));
        kn = *np;
        lr += 16;
        if (lr < r1) {                               // the next load stays on a valid row
            kp += key_step;
            np += norm_step;
        }
    };
    // The products of one tile; the tile's registers are free afterwards.
    auto products = [&](const u32x4 (&bt)[KS], f32x4 (&acc)[NT]) {
        u32x4 b[KS];
        b[0] = dim0 ? bt[0] : u32x4{0u, 0u, 0u, 0u};
        if constexpr (KS == 2) b[1] = dim1 ? bt[1] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            acc[t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                acc[t] = mfma<KT>(ahi[t][ks], b[ks], acc[t]);
                if constexpr (SPLIT) acc[t] = mfma<KT>(alo[t][ks], b[ks], acc[t]);
            }
        }
    };
    // Scores of row r (this lane's key) for every query, then the store
    // (scores) or the filter (survivor keys).
    auto epilogue = [&](int64_t r, const f32x4 (&acc)[NT], float kn) {
        const bool ok = r < r1;
        float v[NT][4];
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[t][i] = acc[t][i];
                if (s.inv_norm) v[t][i] = v[t][i] * kn;
                v[t][i] = v[t][i] * s_qt[16 * t + 4 * grp + i].x;
            }
        if constexpr (!FILTER) {
            if (!ok) return;
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int q = 16 * t + 4 * grp + i;
                    if (q < s.nq) s.scores[(int64_t)q * s.n_rows + r] = v[t][i];
                }
        } else {
            // One float compare per score, all of them (and their threshold
            // reads) before any branch; then a branch per query and key
            // group only where something passed.
            uint64_t bal[NT][4];
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    bal[t][i] = __ballot(ok & !(v[t][i] < s_qt[16 * t + 4 * grp + i].y));
            // Survivors go to this wave's own slots of the query (a slot
            // index from the ballot, no atomic: a returned atomic would make
            // the wave wait for its tiles in flight); a wave with more than
            // kShortSlots survivors for one query appends the rest to the
            // query's overflow list.
            const int64_t orig = r * s.row_step;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (bal[t][i] == 0) continue;
                    const int q = 16 * t + 4 * grp + i;
                    const bool pass = (bal[t][i] >> lane) & 1;
                    const uint32_t gm = (uint32_t)(bal[t][i] >> (16 * grp)) & 0xFFFFu;
                    const int slot = cnt[t][i] + __popc(gm & ((1u << col) - 1u));
                    if (pass && q < s.nq) {
                        const uint64_t key = pack_key(v[t][i], (uint32_t)orig);
                        uint64_t* cq = s.cand + (int64_t)q * s.cap;
                        if (slot < kShortSlots) {
                            cq[wave * kShortSlots + slot] = key;
                        } else {
                            // Rare.  The empty asm keeps this store apart
                            // from the slot store: merged, every survivor
                            // would wait for the atomic's result and with it
                            // for all the tiles in flight.
                            const int pos = atomicAdd(&s.counts[q], 1);
                            cq[pos] = key;
                            __asm__ volatile("" ::: "memory");
                        }
                    }
                    cnt[t][i] += __popc(gm);
                }
            }
        }
    };

    u32x4 buf[kShortDepth][KS];
    float kn[kShortDepth];
    // The first tiles in the loop's own order (keys, then norm, per tile):
    // the wait at the loop head is computed for both ways in, so a
    // different order here would make every iteration wait for more tiles.
#pragma unroll
    for (int u = 0; u < kShortDepth; ++u) {
        load_tile(buf[u], kn[u]);
        __builtin_amdgcn_sched_barrier(0);
    }
    for (int64_t base = r0; base < r1; base += 16 * kShortDepth) {
#pragma unroll
        for (int u = 0; u < kShortDepth; ++u) {
            // The slot's next tile is requested before the epilogue, whose
            // branches would otherwise keep the load behind them.
            f32x4 acc[NT];
            products(buf[u], acc);
            const float knu = kn[u];
            load_tile(buf[u], kn[u]);
            epilogue(base + 16 * u + col, acc, knu);
        }
    }
    if constexpr (FILTER) {
        // Unused slots become padding keys.  Lane col 0 of each group saw
        // every tile its group saw, so its counts are the group's.
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int c0 = __shfl(cnt[t][i], lane & ~15, 64);
                const int q = 16 * t + 4 * grp + i;
                if (q < s.nq && col >= c0 && col < kShortSlots)
                    s.cand[(int64_t)q * s.cap + wave * kShortSlots + col] = 0;
            }
    }
}

// The filtered pass over 64-dim keys with the keys staged in LDS.  Loading
// the matrix-core operand layout straight from HBM (above) reads 64 bytes of
// each of 16 rows per load instruction, a pattern this device serves well
// below its streaming rate, and holds every tile in flight in registers (four
// per wave at most).  Here global_load_lds_dwordx4 moves whole 128-byte rows
// (8 rows per instruction) into a private ring of kRing tile slots per wave,
// kRing - 1 tiles ahead of the products, and each lane reads its operand
// from LDS: lane L = 8p + w of an instruction writes entry w of row p and
// fetches unit (w + p) mod 8 of that row (unit u of row p sits at entry
// (u - p) mod 8, rows 8-15 at entries 64 + ...), so the 8 rows a matrix-core
// read touches in each half fall on 8 distinct 16-byte groups.  A tile's 16
// key norms come the same way (global_load_lds_dword; inner product loads a
// valid dummy word and uses a scale of 1).  Every iteration issues the same
// three loads (tiles past the end reload the last one), so the wait for a
// tile is a fixed count; the loop holds no load into registers, whose waits
// the compiler would take for every load in flight.  The products and the
// filter are those of scan_short_kernel in the same order: the same bits.
// The pass is bound by its per-score instructions, not by HBM; the register
// room the ring frees lets the epilogue take the key scale and the
// row-valid mask once per tile instead of once per score.
constexpr int kRing = 8;           // tile slots per wave
constexpr int kDmaOps = 3;         // loads per tile: two key halves, the norms

template <int KT, int NT, bool SPLIT>
__global__ __launch_bounds__(kShortThreads, 2) void scan_short_lds_kernel(ShortScan s,
                                                                      int64_t rows_per_wave) {
    __shared__ float2 s_qt[64];
    __shared__ __attribute__((aligned(16))) u32x4 s_key[kShortThreads / 64][kRing][128];
    __shared__ __attribute__((aligned(16))) float s_norm[kShortThreads / 64][kRing][64];
    if (threadIdx.x < 64) {
        const int q = threadIdx.x;
        const float th = q < s.nq ? key_score((uint32_t)(s.tau[q] >> 32)) : __builtin_inff();
        s_qt[q] = float2{q < 16 * NT ? s.inv_qn[q] : 0.0f, th};
    }
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t wave = (int64_t)blockIdx.x * (kShortThreads / 64) + wv;
    const int64_t r0 = wave * rows_per_wave;
    if (r0 >= s.n_rows) return;                      // uniform over the wave
    const int64_t r1 = (r0 + rows_per_wave < s.n_rows) ? r0 + rows_per_wave : s.n_rows;
    const int64_t ntiles = (r1 - r0 + 15) / 16;
    const int col = lane & 15, grp = lane >> 4;

    // Query fragments (d = 64: two k-steps), taken into registers before the
    // first LDS load is issued.
    u32x4 ahi[NT][2], alo[NT][2];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const int64_t qoff = (int64_t)(16 * t + col) * 64 + 8 * grp + 32 * ks;
            ahi[t][ks] = *(const u32x4*)(s.qhi + qoff);
            if constexpr (SPLIT) alo[t][ks] = *(const u32x4*)(s.qlo + qoff);
        }
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            asm volatile("" : "+v"(ahi[t][ks]));
            if constexpr (SPLIT) asm volatile("" : "+v"(alo[t][ks]));
        }
    int cnt[NT][4];       // survivors so far per query (same in a 16-lane group)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) cnt[t][i] = 0;

    const uint16_t* keys = (const uint16_t*)s.keys;
    const int64_t rstride = s.row_step * s.ld;
    const bool cosine = s.inv_norm != nullptr;
    const int dp = lane >> 3;                        // row within a load instruction
    const int du = ((lane & 7) + dp) & 7;            // 16-byte unit it fetches
    auto issue = [&](int64_t tile) {
        const int64_t tc = tile < ntiles ? tile : ntiles - 1;
        const int slot = (int)(tile % kRing);
        const int64_t base = r0 + tc * 16;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            int64_t row = base + 8 * i + dp;
            if (row >= r1) row = r1 - 1;
            dma16_nt(keys + row * rstride + du * 8, &s_key[wv][slot][64 * i]);
        }
        int64_t nrow = base + col;
        if (nrow >= r1) nrow = r1 - 1;
        dma4(cosine ? (const void*)(s.inv_norm + nrow * s.row_step) : (const void*)s.inv_qn,
                  &s_norm[wv][slot][0]);
    };
    // Operand entry of this lane in a tile for k-step ks: row col, unit
    // grp + 4 ks.
    auto entry = [&](int ks) {
        const int p = col & 7;
        return 64 * (col >> 3) + 8 * p + (((grp + 4 * ks) - p) & 7);
    };
    const int e0 = entry(0), e1 = entry(1);

#pragma unroll
    for (int t = 0; t < kRing - 1; ++t) issue(t);
    for (int64_t t = 0; t < ntiles; ++t) {
        wait_vmcnt<(kRing - 2) * kDmaOps>();           // tile t is in LDS
        issue(t + kRing - 1);                       // the slot read at t - 1
        const int slot = (int)(t % kRing);
        const u32x4 b0 = s_key[wv][slot][e0], b1 = s_key[wv][slot][e1];
        const float kn = s_norm[wv][slot][col];
        f32x4 acc[NT];
#pragma unroll
        for (int q = 0; q < NT; ++q) {
            acc[q] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            acc[q] = mfma<KT>(ahi[q][0], b0, acc[q]);
            if constexpr (SPLIT) acc[q] = mfma<KT>(alo[q][0], b0, acc[q]);
            acc[q] = mfma<KT>(ahi[q][1], b1, acc[q]);
            if constexpr (SPLIT) acc[q] = mfma<KT>(alo[q][1], b1, acc[q]);
        }
        const int64_t r = r0 + t * 16 + col;
        // Inner product scales by 1 (x * 1 is x: the same bits as no scale).
        const float ks = cosine ? kn : 1.0f;
        const uint64_t okm = __ballot(r < r1);
        float v[NT][4];
#pragma unroll
        for (int q = 0; q < NT; ++q)
#pragma unroll
            for (int i = 0; i < 4; ++i) v[q][i] = (acc[q][i] * ks) * s_qt[16 * q + 4 * grp + i].x;
        uint64_t bal[NT][4];
#pragma unroll
        for (int q = 0; q < NT; ++q)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                bal[q][i] = __ballot(!(v[q][i] < s_qt[16 * q + 4 * grp + i].y)) & okm;
        const int64_t orig = r * s.row_step;
#pragma unroll
        for (int q = 0; q < NT; ++q) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (bal[q][i] == 0) continue;
                const int qi = 16 * q + 4 * grp + i;
                const bool pass = (bal[q][i] >> lane) & 1;
                const uint32_t gm = (uint32_t)(bal[q][i] >> (16 * grp)) & 0xFFFFu;
                const int slot_i = cnt[q][i] + __popc(gm & ((1u << col) - 1u));
                if (pass && qi < s.nq) {
                    const uint64_t key = pack_key(v[q][i], (uint32_t)orig);
                    uint64_t* cq = s.cand + (int64_t)qi * s.cap;
                    if (slot_i < kShortSlots) {
                        cq[wave * kShortSlots + slot_i] = key;
                    } else {
                        const int pos = atomicAdd(&s.counts[qi], 1);
                        cq[pos] = key;
                        __asm__ volatile("" ::: "memory");
                    }
                }
                cnt[q][i] += __popc(gm);
            }
        }
    }
    wait_vmcnt<0>();
    // Unused slots become padding keys (lane col 0 of each group saw every
    // tile its group saw).
#pragma unroll
    for (int q = 0; q < NT; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c0 = __shfl(cnt[q][i], lane & ~15, 64);
            const int qi = 16 * q + 4 * grp + i;
            if (qi < s.nq && col >= c0 && col < kShortSlots)
                s.cand[(int64_t)qi * s.cap + wave * kShortSlots + col] = 0;
        }
}

__global__ void short_tau_kernel(const int64_t* __restrict__ ids, const float* __restrict__ scores,
                                 int nq, int k, int64_t row_step, int32_t slot_area,
                                 const float* __restrict__ margin, uint64_t* __restrict__ tau,
                                 int32_t* __restrict__ counts) {
    const int q = blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= nq) return;
    const int64_t id = ids[(int64_t)q * k + (k - 1)];
    // A sample shorter than k leaves a padding id: then every row passes.
    // With approximate scores the threshold is lowered by the margin.
    float s = scores[(int64_t)q * k + (k - 1)];
    if (margin) s = s - margin[q];
    tau[q] = id < 0 ? 0ull : pack_key(s, (uint32_t)(id * row_step));
    counts[q] = slot_area;          // overflow entries follow the wave slots
}

template <int KT, int NT, int KS, bool SPLIT, bool FILTER>
hipError_t launch_variant(const ShortScan& s, hipStream_t stream) {
    auto kern = scan_short_kernel<KT, NT, KS, SPLIT, FILTER>;
    const int64_t rpw = short_rows_per_wave(s.n_rows);
    const int64_t waves = (s.n_rows + rpw - 1) / rpw;
    const int64_t blocks = (waves + (kShortThreads / 64) - 1) / (kShortThreads / 64);
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kShortThreads), 0, stream, s, rpw);
    return hipGetLastError();
}

template <int KT, int NT, int KS>
hipError_t launch_mode(const ShortScan& s, hipStream_t stream) {
    const bool filter = s.cand != nullptr;
    if constexpr (KS == 2) {
        // 64-dim keys, filtered: the LDS-staged pass (16-byte aligned rows).
        if (filter && s.d == 64 && ((uintptr_t)s.keys % 16) == 0 && (s.row_step * s.ld) % 8 == 0) {
            const int64_t rpw = short_rows_per_wave(s.n_rows);
            const int64_t waves = (s.n_rows + rpw - 1) / rpw;
            const int64_t blocks = (waves + (kShortThreads / 64) - 1) / (kShortThreads / 64);
            if (s.split)
                hipLaunchKernelGGL((scan_short_lds_kernel<KT, NT, true>), dim3((unsigned)blocks),
                                   dim3(kShortThreads), 0, stream, s, rpw);
            else
                hipLaunchKernelGGL((scan_short_lds_kernel<KT, NT, false>), dim3((unsigned)blocks),
                                   dim3(kShortThreads), 0, stream, s, rpw);
            return hipGetLastError();
        }
    }
    if (s.split)
        return filter ? launch_variant<KT, NT, KS, true, true>(s, stream)
                      : launch_variant<KT, NT, KS, true, false>(s, stream);
    return filter ? launch_variant<KT, NT, KS, false, true>(s, stream)
                  : launch_variant<KT, NT, KS, false, false>(s, stream);
}

template <int KT, int KS>
hipError_t launch_tiles(const ShortScan& s, hipStream_t stream) {
    switch ((s.nq + 15) / 16) {
        case 1: return launch_mode<KT, 1, KS>(s, stream);
        case 2: return launch_mode<KT, 2, KS>(s, stream);
        case 3: return launch_mode<KT, 3, KS>(s, stream);
        default: return launch_mode<KT, 4, KS>(s, stream);
    }
}

}  // namespace

int64_t short_rows_per_wave(int64_t n_rows) {
    // Two resident waves per SIMD (the kernels' register use allows two).
    const int64_t waves_max = (int64_t)device_cus() * 8;
    int64_t rpw = (n_rows + waves_max - 1) / waves_max;
    return (rpw + 16 * kShortDepth - 1) / (16 * kShortDepth) * (16 * kShortDepth);
}

int64_t short_scan_waves(int64_t n_rows) {
    const int64_t rpw = short_rows_per_wave(n_rows);
    return (n_rows + rpw - 1) / rpw;
}

hipError_t launch_scan_short(const ShortScan& s, hipStream_t stream) {
    const bool two = s.d > 32;
    if (s.key_dtype == DT_BF16)
        return two ? launch_tiles<DT_BF16, 2>(s, stream) : launch_tiles<DT_BF16, 1>(s, stream);
    return two ? launch_tiles<DT_F16, 2>(s, stream) : launch_tiles<DT_F16, 1>(s, stream);
}

hipError_t launch_short_tau(const int64_t* ids, const float* scores, int nq, int k,
                            int64_t row_step, int32_t slot_area, const float* margin,
                            uint64_t* tau, int32_t* counts, hipStream_t stream) {
    hipLaunchKernelGGL(short_tau_kernel, dim3((unsigned)((nq + 63) / 64)), dim3(64), 0, stream,
                       ids, scores, nq, k, row_step, slot_area, margin, tau, counts);
    return hipGetLastError();
}

}  // namespace sense
