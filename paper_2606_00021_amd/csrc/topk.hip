// Per-query top-k of the similarity scores (Sec. 3.1 Eq. 3: the retriever
// returns the N most relevant continuations; Sec. 3.2 Eq. 7 "top-N'") and
// the gather of each hit's continuation into the draft batch (the (k_i, s_i)
// pairs of Sec. 3.2).
//
// Order: score descending, then row index ascending.  Each (score, row) pair
// is packed into one unique 64-bit key (order-preserving score bits in the
// high word, the complemented row in the low word), so "top-k" is "the k
// largest keys" and ties need no special handling.
//
// Selection is hierarchical.  A block of 512 threads takes a chunk of 8192
// keys into registers (16 per thread; a single chunk of at most 4096 keys
// takes 8 per thread, since every phase costs its per-thread key loop).
// The block is one compute unit, so every per-key instruction counts.  One
// reduction gives the number of real (non-padding) keys and the AND and OR
// of them: the bits above the highest bit where they differ are shared by
// all, so the radix select starts right below them (survivors of a level
// share their sign and most of their exponent, which a fixed top-down start
// would spend a whole pass on).  For a chunk of raw scores the AND and OR
// come from the score words alone, the row words being a contiguous range.
// A chunk of raw scores holds both signs, so the first level also bounds the
// k-th largest key from below by the smallest of k or more group maxima and
// starts below the bits that this bound and the largest key share: every
// key of the top k lies between them.  Each pass builds a 256-bin LDS
// histogram of the next 8-bit digit among the keys that still match the
// chosen prefix, then one wave totals the waves' histograms and finds the
// digit holding the k-th key with a suffix scan; the loop stops as soon as
// that digit's bucket is taken whole.  The taken keys are compacted by ballot prefix sums (no atomics).
// The k survivors of every chunk form the next level's input until one
// chunk remains; its keys are put in order by rank (each key counts the
// keys above it, all reads LDS broadcasts) and written out together with
// the gathered continuations.
#include "internal.h"

namespace sense {
namespace {

constexpr int kThreads = 512;

struct SelectState {
    uint64_t prefix;
    uint64_t mask;
};

constexpr int kWaves = kThreads / 64;
constexpr int kRankMax = 256;   // final orders up to this many keys by rank, more by bitonic sort
constexpr int kPer = kSelectChunk / kThreads;   // keys per thread

// Real keys of the block (non-zero; a candidate buffer may hold padding keys
// anywhere, so a chunk's length alone does not tell) and the AND / OR of
// them.  With BOUND, also the score words (high 32 bits) of the largest key
// and of a lower bound on the kk-th largest: the threads are cut into
// G >= kk groups of g consecutive lanes, and `low` is the smallest of the G
// group maxima.  Those maxima are G distinct keys (or one is the padding key
// and low = 0), so at least kk keys are >= low; the score word of a maximum
// (minimum) is the maximum (minimum) of the score words.  All threads of the
// block must call it.
struct ChunkStats {
    uint32_t nz;
    uint64_t all_and, any_or;
    uint32_t low32, high32;
};

struct StatsLds {
    uint32_t* nzw;
    uint64_t* andw;
    uint64_t* orw;
    uint32_t* loww;
    uint32_t* highw;
};

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}

// The group-maxima bound of the comment above from each lane's largest
// score word mx: hi = the largest mx of the wave, lo = the smallest of its
// group maxima (wave-uniform results).  Group size g: the largest power
// of two <= 64 with T / g >= kk; none (lo = 0) when kk > T.  One max ladder
// over groups of 2, 4, ..., 64 lanes (quad swaps, half-row and row mirrors,
// then xor 16 and 32), keeping the group maxima at size g; then the min
// ladder of those.
template <int T>
__device__ __forceinline__ void group_bound(uint32_t mx, int kk, uint32_t* lo_out,
                                            uint32_t* hi_out) {
    const int gq = T / (kk > 0 ? kk : 1);
    const int g = gq >= 64 ? 64 : (gq > 0 ? 1 << (31 - __clz(gq)) : 0);
    uint32_t v = mx, gm = (g == 1) ? mx : 0u;
    auto mxs = [](uint32_t x, uint32_t y) { return x > y ? x : y; };
    auto mns = [](uint32_t x, uint32_t y) { return x < y ? x : y; };
    v = mxs(v, dpp_u<0xB1>(v));  gm = (g == 2) ? v : gm;
    v = mxs(v, dpp_u<0x4E>(v));  gm = (g == 4) ? v : gm;
    v = mxs(v, dpp_u<0x141>(v)); gm = (g == 8) ? v : gm;
    v = mxs(v, dpp_u<0x140>(v)); gm = (g == 16) ? v : gm;
    v = mxs(v, (uint32_t)__shfl_xor((int)v, 16, 64)); gm = (g == 32) ? v : gm;
    v = mxs(v, (uint32_t)__shfl_xor((int)v, 32, 64)); gm = (g == 64) ? v : gm;
    uint32_t lo = gm;
    lo = mns(lo, dpp_u<0xB1>(lo));
    lo = mns(lo, dpp_u<0x4E>(lo));
    lo = mns(lo, dpp_u<0x141>(lo));
    lo = mns(lo, dpp_u<0x140>(lo));
    lo = mns(lo, (uint32_t)__shfl_xor((int)lo, 16, 64));
    lo = mns(lo, (uint32_t)__shfl_xor((int)lo, 32, 64));
    *lo_out = lo;
    *hi_out = v;
}

// Block-wide combination of the per-wave statistics (wave-uniform inputs).
template <int T, bool BOUND>
__device__ __forceinline__ ChunkStats combine_waves(uint32_t nz, uint64_t a, uint64_t o,
                                                    uint32_t lo, uint32_t hi,
                                                    const StatsLds& L) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    if (lane == 0) {
        L.nzw[wv] = nz;
        L.andw[wv] = a;
        L.orw[wv] = o;
        if constexpr (BOUND) {
            L.loww[wv] = lo;
            L.highw[wv] = hi;
        }
    }
    __syncthreads();
    ChunkStats r{0u, ~0ull, 0ull, ~0u, 0u};
#pragma unroll
    for (int w = 0; w < T / 64; ++w) {
        r.nz += L.nzw[w];
        r.all_and &= L.andw[w];
        r.any_or |= L.orw[w];
        if constexpr (BOUND) {
            r.low32 = L.loww[w] < r.low32 ? L.loww[w] : r.low32;
            r.high32 = L.highw[w] > r.high32 ? L.highw[w] : r.high32;
        }
    }
    if constexpr (!BOUND) r.low32 = r.high32 = 0u;
    return r;
}

template <int T, int P, bool BOUND>
__device__ ChunkStats chunk_stats(const uint64_t (&key)[P], int kk, const StatsLds& L) {
    uint32_t nz = 0;
    uint64_t a = ~0ull, o = 0ull;
    uint32_t mx = 0u;
#pragma unroll
    for (int e = 0; e < P; ++e) {
        nz += (uint32_t)__popcll(__ballot(key[e] != 0));
        if (key[e] != 0) {
            a &= key[e];
            o |= key[e];
        }
        if constexpr (BOUND) {
            const uint32_t h = (uint32_t)(key[e] >> 32);
            mx = h > mx ? h : mx;
        }
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        a &= __shfl_xor(a, off, 64);
        o |= __shfl_xor(o, off, 64);
    }
    uint32_t lo = 0u, hi = 0u;
    if constexpr (BOUND) group_bound<T>(mx, kk, &lo, &hi);
    return combine_waves<T, BOUND>(nz, a, o, lo, hi, L);
}

// chunk_stats with the bound for a chunk of raw scores, rows start ..
// start + len - 1 (len >= 1), without a conditional per key.  sw[e] is the
// score word of slot e's row, past the chunk a copy of the last row's (a
// copy changes no AND or OR); the high word of key[e] is 0 past the chunk
// (for the maxima, which must be distinct keys).  Every slot before len is
// a real key.  The row words are the complements of a contiguous range of
// indices: above the highest bit where the first and the last differ all
// share their bits, and below it both values occur at every bit (the range
// holds the two indices on either side of the carry into that bit), so
// their AND and OR follow from the two ends.
template <int T, int P>
__device__ ChunkStats score_stats(const uint32_t (&sw)[P], const uint64_t (&key)[P], int kk,
                                  int64_t start, int len, const StatsLds& L) {
    uint32_t a = ~0u, o = 0u, mx = 0u;
#pragma unroll
    for (int e = 0; e < P; ++e) {
        a &= sw[e];
        o |= sw[e];
        const uint32_t h = (uint32_t)(key[e] >> 32);
        mx = h > mx ? h : mx;
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        a &= (uint32_t)__shfl_xor((int)a, off, 64);
        o |= (uint32_t)__shfl_xor((int)o, off, 64);
    }
    uint32_t lo, hi;
    group_bound<T>(mx, kk, &lo, &hi);
    ChunkStats r = combine_waves<T, true>(0u, (uint64_t)a << 32, (uint64_t)o << 32, lo, hi, L);
    const uint32_t first = 0xFFFFFFFFu - (uint32_t)start;
    const uint32_t x = first ^ (0xFFFFFFFFu - (uint32_t)(start + len - 1));
    const uint32_t below = x ? (0xFFFFFFFFu >> __clz(x)) : 0u;   // bits up to the highest of x
    r.nz = (uint32_t)len;
    r.all_and |= first & ~below;
    r.any_or |= first | below;
    return r;
}

// Finds prefix/mask such that exactly `need` of the block's keys (P per
// thread, held in registers; unused slots hold the padding key 0) satisfy
// (key & mask) >= prefix.  Requires 1 <= need < cs.nz (the number of real
// keys).  All threads of the block must call it.
//
// Digits of up to 8 bits from the highest bit where the real keys differ; a
// pass stops the search as soon as the digit holding the need-th key is
// taken whole.  Each wave counts into its own 256-bin LDS histogram with
// plain LDS atomics (starting below the shared bits spreads the keys over
// the digit values, so same-address collisions inside an instruction stay
// few).
template <int T, int P, bool BOUND>
__device__ SelectState radix_select(const uint64_t (&key)[P], int need, const ChunkStats& cs,
                                    uint32_t* s_hist, uint32_t* s_info) {
    const int tid = threadIdx.x;
    const int wv = tid >> 6;
    uint32_t* my = s_hist + wv * 256;
    const uint64_t diff = cs.all_and ^ cs.any_or;
    if (diff == 0) return SelectState{cs.all_and, ~0ull};   // every real key is the same
    // Bits above hb are common to every real key (2 << 63 wraps to 0: no
    // bits).  With BOUND they are also common to every key in [low, high],
    // which holds the need largest: the score-word bits above the highest
    // one where low and high differ (the whole score word if none does).
    int hb = 63 - __clzll((long long)diff);
    if constexpr (BOUND) {
        const uint32_t span = cs.low32 ^ cs.high32;
        const int hs = span ? 63 - __clz(span) : 31;
        hb = hs < hb ? hs : hb;
    }
    uint64_t mask = ~((2ull << hb) - 1ull);
    // Above bit 31 the bits are the largest key's score word; below, every
    // real key shares them (hb < 31 only when all share the score word).
    uint64_t prefix = (BOUND ? (((uint64_t)cs.high32 << 32) | (cs.all_and & 0xFFFFFFFFull))
                             : cs.all_and) & mask;
    for (int b = tid; b < (T / 64) * 256; b += T) s_hist[b] = 0;
    __syncthreads();
    for (int hi = hb; hi >= 0; hi -= 8) {
        const int lo = hi >= 7 ? hi - 7 : 0;
        const uint32_t dmask = (1u << (hi - lo + 1)) - 1u;
#pragma unroll
        for (int e = 0; e < P; ++e) {
            const bool act = (key[e] & mask) == prefix;
            const uint32_t dg = (uint32_t)(key[e] >> lo) & dmask;
            if (act) atomicAdd(&my[dg], 1u);
        }
        __syncthreads();
        // Wave 0: the totals of its lane's four digits over the waves'
        // histograms (16-byte LDS reads; the histograms cleared for the next
        // pass), then the digit holding the need-th key by a suffix scan.
        if (tid < 64) {
            const int l = tid;
            typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
            u32x4_t h = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int w = 0; w < T / 64; ++w) {
                u32x4_t* p = (u32x4_t*)(s_hist + w * 256 + 4 * l);
                h += *p;
                *p = u32x4_t{0u, 0u, 0u, 0u};
            }
            const uint32_t h0 = h[0], h1 = h[1], h2 = h[2], h3 = h[3];
            const uint32_t local = h0 + h1 + h2 + h3;
            // inclusive suffix sum over lanes l..63 (higher digits)
            uint32_t incl = local;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const uint32_t t = __shfl_down(incl, off, 64);
                if (l + off < 64) incl += t;
            }
            uint32_t above = incl - local;
            if (above < (uint32_t)need && (uint32_t)need <= incl) {
                const uint32_t hs[4] = {h0, h1, h2, h3};
                for (int j = 3; j >= 0; --j) {
                    if (above + hs[j] >= (uint32_t)need) {
                        s_info[0] = (uint32_t)(4 * l + j);
                        s_info[1] = above;
                        s_info[2] = hs[j];
                        break;
                    }
                    above += hs[j];
                }
            }
        }
        __syncthreads();
        // Every thread reads s_info before any thread passes the next pass's
        // first barrier, after which wave 0 may rewrite it.
        const uint32_t digit = s_info[0], above = s_info[1], in_bucket = s_info[2];
        need -= (int)above;
        prefix |= (uint64_t)digit << lo;
        mask |= (uint64_t)dmask << lo;
        if ((int)in_bucket == need) break;
    }
    __syncthreads();
    return SelectState{prefix, mask};
}

// Writes the block's taken keys, those with (key & tmask) >= tpre, to
// dst[0 .. min(taken, cap)) in some order, positions from ballot prefix sums
// (each wave's count, then its lanes' ranks inside each key slot); returns
// the number taken (all threads).  One masked compare per key and slot; a
// slot where the wave takes nothing is skipped on the scalar unit.
template <int T, int P>
__device__ uint32_t compact_taken(const uint64_t (&key)[P], uint64_t tmask, uint64_t tpre,
                                  uint64_t* dst, int cap, uint32_t* s_wc) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    uint32_t mine = 0;
#pragma unroll
    for (int e = 0; e < P; ++e) mine += (uint32_t)__popcll(__ballot((key[e] & tmask) >= tpre));
    if (lane == 0) s_wc[wv] = mine;
    __syncthreads();
    uint32_t base = 0, total = 0;
#pragma unroll
    for (int w = 0; w < T / 64; ++w) {
        const uint32_t c = s_wc[w];
        base += (w < wv) ? c : 0u;
        total += c;
    }
    if (mine != 0u) {                                  // uniform over the wave
        const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
        for (int e = 0; e < P; ++e) {
            const bool t = (key[e] & tmask) >= tpre;
            const uint64_t m = __ballot(t);
            if (m != 0ull) {
                const uint32_t pos = base + (uint32_t)__popcll(m & below);
                if (t && pos < (uint32_t)cap) dst[pos] = key[e];
                base += (uint32_t)__popcll(m);
            }
        }
    }
    return total;
}

// The final level's output: the nt taken keys of s_sel (nt <= k) in order
// by rank (k <= kRankMax: each key counts the keys above it, LDS broadcast
// reads) or by a bitonic network, then ids, scores and the gathered
// continuations of query q; padding keys give id -1.  All threads of the
// block must call it.
template <int T>
__device__ void final_output(uint64_t* s_sel, uint64_t* s_sorted, int nt, int k, int q,
                             int64_t* __restrict__ out_ids, float* __restrict__ out_scores,
                             int32_t* __restrict__ out_drafts, int32_t* __restrict__ out_draft_len,
                             const int32_t* __restrict__ spans, const int32_t* __restrict__ span_len,
                             int max_span, int64_t span_stride) {
    const int tid = threadIdx.x;
    int p = 1;
    while (p < nt) p <<= 1;
    __syncthreads();
    const uint64_t* sorted = s_sorted;
    if (p <= kRankMax) {
        // Rank of each taken key among the taken ones (ties, impossible
        // for distinct (score, row) keys, by position): its place in the
        // output.  g = T / p threads share a key's count, each over every
        // g-th key, and add their parts in LDS.
        __shared__ int s_rank[kRankMax];
        for (int i = tid; i < nt; i += T) s_rank[i] = 0;
        __syncthreads();
        const int g = T / p;
        const int i = tid / g, part = tid - (tid / g) * g;
        const uint64_t ki = i < nt ? s_sel[i] : 0ull;
        if (i < nt) {
            int c = 0;
            for (int j = part; j < nt; j += g) {
                const uint64_t kj = s_sel[j];
                c += (kj > ki) | ((kj == ki) & (j < i));
            }
            if (c) atomicAdd(&s_rank[i], c);
        }
        __syncthreads();
        if (i < nt && part == 0) s_sorted[s_rank[i]] = ki;
        for (int r = nt + tid; r < k; r += T) s_sorted[r] = 0;
    } else {
        // padding keys up to the sort size and up to k (read as output)
        for (int r = nt + tid; r < (p > k ? p : k); r += T) s_sel[r] = 0;
        __syncthreads();
        bitonic_desc<T>(s_sel, p);
        sorted = s_sel;
    }
    __syncthreads();
    for (int r = tid; r < k; r += T) {
        const uint64_t key = sorted[r];
        out_ids[(int64_t)q * k + r] = key == 0 ? -1 : (int64_t)key_row(key);
        if (out_scores) out_scores[(int64_t)q * k + r] = key_score((uint32_t)(key >> 32));
    }
    if (out_drafts || out_draft_len) {
        for (int t = tid; t < k * max_span; t += T) {
            const int r = t / max_span, j = t - r * max_span;
            const uint64_t key = sorted[r];
            // A padding key (0) surfaces only when fewer than k
            // candidates exist (an inverted-file search of short lists):
            // id -1, score NaN, an empty draft.  Its loads read row 0 so that
            // the length and the token are both in flight at once.
            const int64_t id = key == 0 ? 0 : (int64_t)key_row(key);
            const int tok = out_drafts ? spans[id * span_stride + j] : 0;
            int len_r = (key == 0) ? 0 : (span_len ? span_len[id] : max_span);
            len_r = len_r < 0 ? 0 : (len_r > max_span ? max_span : len_r);
            const int64_t o = ((int64_t)q * k + r);
            if (out_drafts)
                out_drafts[o * max_span + j] = (j < len_r) ? tok : -1;
            if (out_draft_len && j == 0) out_draft_len[o] = len_r;
        }
    }
}

// One block per (chunk, query).  FROM_SCORES: input is the fp32 score matrix
// (nq x count, row index = position); otherwise packed keys (nq x count).
// FINAL: exactly one chunk per query; writes sorted ids/scores and drafts.
// P keys per thread: chunks of kThreads * P keys (kSelectChunk for P = 16;
// a smaller P serves a single chunk of fewer keys with less work).
template <bool FROM_SCORES, bool FINAL, int P>
__global__ __launch_bounds__(kThreads) void select_kernel(
    const float* __restrict__ scores, const uint64_t* __restrict__ in_keys, int64_t count,
    int k, uint64_t* __restrict__ out_keys, int64_t* __restrict__ out_ids,
    float* __restrict__ out_scores, int32_t* __restrict__ out_drafts,
    int32_t* __restrict__ out_draft_len, const int32_t* __restrict__ spans,
    const int32_t* __restrict__ span_len, int max_span, int64_t span_stride) {
    __shared__ uint64_t s_sel[kMaxK];
    __shared__ uint64_t s_sorted[FINAL ? kMaxK : 1];
    __shared__ __align__(16) uint32_t s_hist[kWaves * 256];   // read 16 bytes at a time
    __shared__ uint32_t s_info[4];
    __shared__ uint32_t s_nzw[kWaves], s_wc[kWaves];
    __shared__ uint64_t s_andw[kWaves], s_orw[kWaves];
    __shared__ uint32_t s_loww[kWaves], s_highw[kWaves];

    constexpr int CH = kThreads * P;
    const int tid = threadIdx.x;
    const int q = blockIdx.y;
    const int64_t start = (int64_t)blockIdx.x * CH;
    const int64_t remain = count - start;
    const int len = (int)(remain < CH ? remain : CH);
    const int kk = k < CH ? k : CH;

    // Key i of the chunk is held by thread i % kThreads; slots past the chunk
    // hold the padding key 0.  Scores are loaded unconditionally (positions
    // past the chunk re-read its last one, a chunk is never empty here) so
    // that all loads are in flight at once: a load under a branch makes the
    // thread wait for it before issuing the next.
    // The group-maxima bound pays where a chunk holds raw scores of both
    // signs (its keys share no leading bits), first levels and single-chunk
    // finals alike; later levels hold survivors that already share them.
    constexpr bool kBound = FROM_SCORES;
    const StatsLds lds{s_nzw, s_andw, s_orw, s_loww, s_highw};
    uint64_t key[P];
    ChunkStats cs;
    if constexpr (FROM_SCORES) {
        const float* src = scores + (int64_t)q * count + start;
        const int last = len > 0 ? len - 1 : 0;
        float sv[P];
#pragma unroll
        for (int e = 0; e < P; ++e) {
            const int i = tid + e * kThreads;
            sv[e] = src[i < len ? i : last];
        }
        uint32_t sw[P];
#pragma unroll
        for (int e = 0; e < P; ++e) {
            const int i = tid + e * kThreads;
            sw[e] = score_key(sv[e]);
            key[e] = i < len ? (((uint64_t)sw[e] << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)(start + i)))
                             : 0ull;
        }
        cs = score_stats<kThreads, P>(sw, key, kk, start, len, lds);
    } else {
#pragma unroll
        for (int e = 0; e < P; ++e) {
            const int i = tid + e * kThreads;
            key[e] = i < len ? in_keys[(int64_t)q * count + start + i] : 0;
        }
        cs = chunk_stats<kThreads, P, kBound>(key, kk, lds);
    }

    // Keys taken: every real (non-zero) one if there are no more than kk,
    // else the kk largest (then more than kk keys are real, as the radix
    // select needs); both as (key & mask) >= prefix.
    SelectState st{1ull, ~0ull};
    const bool all = cs.nz <= (uint32_t)kk;
    if (!all) st = radix_select<kThreads, P, kBound>(key, kk, cs, s_hist, s_info);

    if constexpr (!FINAL) {
        uint64_t* out = out_keys + ((int64_t)q * gridDim.x + blockIdx.x) * kk;
        const uint32_t tot = compact_taken<kThreads, P>(key, st.mask, st.prefix, out, kk, s_wc);
        const int nt = (int)tot < kk ? (int)tot : kk;
        for (int i = nt + tid; i < kk; i += kThreads) out[i] = 0;  // padding key
    } else {
        const uint32_t tot = compact_taken<kThreads, P>(key, st.mask, st.prefix, s_sel, kk, s_wc);
        const int nt = (int)tot < kk ? (int)tot : kk;
        final_output<kThreads>(s_sel, s_sorted, nt, k, q, out_ids, out_scores, out_drafts,
                               out_draft_len, spans, span_len, max_span, span_stride);
    }
}

// One block per query over a key list whose length is a per-query count on
// the device (candidate buffers: most of the capacity is unused): rounds of
// kStreamThreads * P keys, each holding the running top k and the next new
// keys, reduced to the top k by the same radix select; then the final
// output.  P (keys per thread) is chosen per query from its count, so a short
// list is walked with less work; a count that fits one round of the largest
// P is one round, and any count is exact.
constexpr int kStreamThreads = 1024;
constexpr int kStreamPer = kPer;                       // the largest P

struct StreamLds {
    uint32_t* s_hist;
    uint32_t* s_info;
    uint32_t* s_nzw;
    uint32_t* s_wc;
    uint64_t* s_andw;
    uint64_t* s_orw;
};

template <int P>
__device__ int stream_rounds(const uint64_t* __restrict__ src, int64_t count, int64_t cnt_q,
                             int kk, uint64_t* s_sel, const StreamLds& L) {
    constexpr int R = kStreamThreads * P;              // keys per round
    const int tid = threadIdx.x;
    int nt = 0;                                        // running top keys in s_sel
    int64_t pos = 0;
    do {
        const int64_t left = cnt_q - pos;
        const int take = (int)((R - nt) < left ? (R - nt) : left);
        // New keys on clamped positions (no branch around a load), the
        // running ones from LDS.
        uint64_t key[P];
#pragma unroll
        for (int e = 0; e < P; ++e) {
            const int i = tid + e * kStreamThreads;
            const int64_t j = pos + (i - nt);
            const int64_t jc = j < 0 ? 0 : (j < count ? j : count - 1);
            key[e] = src[jc];
        }
#pragma unroll
        for (int e = 0; e < P; ++e) {
            const int i = tid + e * kStreamThreads;
            if (i < nt) key[e] = s_sel[i];
            else if (i - nt >= take) key[e] = 0;
        }
        __syncthreads();                               // s_sel read before it is rewritten
        const ChunkStats cs = chunk_stats<kStreamThreads, P, false>(
            key, kk, StatsLds{L.s_nzw, L.s_andw, L.s_orw, nullptr, nullptr});
        SelectState st{1ull, ~0ull};                   // all real keys, as above
        const bool all = cs.nz <= (uint32_t)kk;
        if (!all)
            st = radix_select<kStreamThreads, P, false>(key, kk, cs, L.s_hist, L.s_info);
        const uint32_t tot =
            compact_taken<kStreamThreads, P>(key, st.mask, st.prefix, s_sel, kk, L.s_wc);
        nt = (int)tot < kk ? (int)tot : kk;
        pos += take;
        __syncthreads();                               // s_sel complete for the next round
    } while (pos < cnt_q);
    return nt;
}

__global__ __launch_bounds__(kStreamThreads) void select_stream_kernel(
    const uint64_t* __restrict__ in_keys, int64_t count, int k,
    const int32_t* __restrict__ dev_count, int64_t* __restrict__ out_ids,
    float* __restrict__ out_scores, int32_t* __restrict__ out_drafts,
    int32_t* __restrict__ out_draft_len, const int32_t* __restrict__ spans,
    const int32_t* __restrict__ span_len, int max_span, int64_t span_stride) {
    constexpr int W = kStreamThreads / 64;
    __shared__ uint64_t s_sel[kMaxK];
    __shared__ uint64_t s_sorted[kMaxK];
    __shared__ __align__(16) uint32_t s_hist[W * 256];        // read 16 bytes at a time
    __shared__ uint32_t s_info[4];
    __shared__ uint32_t s_nzw[W], s_wc[W];
    __shared__ uint64_t s_andw[W], s_orw[W];
    const StreamLds L{s_hist, s_info, s_nzw, s_wc, s_andw, s_orw};
    const int q = blockIdx.x;
    const int kk = k;                                  // k <= kMaxK < kStreamThreads * 4
    int64_t cnt_q = dev_count ? (int64_t)dev_count[q] : count;
    cnt_q = cnt_q < 0 ? 0 : (cnt_q > count ? count : cnt_q);
    const uint64_t* src = in_keys + (int64_t)q * count;
    // The branch is uniform over the block.
    int nt;
    if (cnt_q <= (int64_t)kStreamThreads * 4)
        nt = stream_rounds<4>(src, count, cnt_q, kk, s_sel, L);
    else if (cnt_q <= (int64_t)kStreamThreads * 8)
        nt = stream_rounds<8>(src, count, cnt_q, kk, s_sel, L);
    else
        nt = stream_rounds<kStreamPer>(src, count, cnt_q, kk, s_sel, L);
    final_output<kStreamThreads>(s_sel, s_sorted, nt, k, q, out_ids, out_scores, out_drafts,
                                 out_draft_len, spans, span_len, max_span, span_stride);
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// The final level over one chunk of keys (count <= kSelectChunk): eight
// keys per thread when they fit.
void launch_final_keys(const uint64_t* keys, int64_t count, int nq, int k, const int32_t* spans,
                       const int32_t* span_len, int max_span, int64_t span_stride,
                       int64_t* out_ids, float* out_scores, int32_t* out_drafts,
                       int32_t* out_draft_len, hipStream_t stream) {
    if (count <= (int64_t)kThreads * 8)
        hipLaunchKernelGGL((select_kernel<false, true, 8>), dim3(1, nq), dim3(kThreads), 0,
                           stream, nullptr, keys, count, k, nullptr, out_ids, out_scores,
                           out_drafts, out_draft_len, spans, span_len, max_span, span_stride);
    else
        hipLaunchKernelGGL((select_kernel<false, true, kPer>), dim3(1, nq), dim3(kThreads), 0,
                           stream, nullptr, keys, count, k, nullptr, out_ids, out_scores,
                           out_drafts, out_draft_len, spans, span_len, max_span, span_stride);
}

}  // namespace

// One of the two key buffers of the selection levels, 256-byte rounded.
static size_t key_buffer_bytes(int64_t n, int nq, int k) {
    const int64_t chunks = ceil_div(n, kSelectChunk);
    const int64_t kk = k < kSelectChunk ? k : kSelectChunk;
    return ((size_t)nq * (size_t)chunks * (size_t)kk * sizeof(uint64_t) + 255) / 256 * 256;
}

size_t topk_workspace_bytes(int64_t n, int nq, int k) {
    const int64_t chunks = ceil_div(n, kSelectChunk);
    if (chunks <= 1) return 0;
    const int64_t kk = k < kSelectChunk ? k : kSelectChunk;
    const size_t one = (size_t)nq * (size_t)chunks * (size_t)kk * sizeof(uint64_t);
    return 2 * ((one + 255) / 256 * 256);                // the two key buffers
}

hipError_t launch_topk_gather(const float* scores, int64_t n, int nq, int k,
                              const int32_t* spans, const int32_t* span_len, int max_span,
                              int64_t span_stride, int64_t* out_ids, float* out_scores, int32_t* out_drafts,
                              int32_t* out_draft_len, void* workspace, hipStream_t stream) {
    const int64_t kk = k < kSelectChunk ? k : kSelectChunk;
    int64_t chunks = ceil_div(n, kSelectChunk);
    if (chunks <= 2) {
        // One block: up to kThreads * 8 scores take eight per thread, up to
        // two chunks' worth 32 (one launch instead of a level and a final).
        if (n > kSelectChunk) {
            hipLaunchKernelGGL((select_kernel<true, true, 2 * kPer>), dim3(1, nq), dim3(kThreads),
                               0, stream, scores, nullptr, n, k, nullptr, out_ids, out_scores,
                               out_drafts, out_draft_len, spans, span_len, max_span, span_stride);
            return hipGetLastError();
        }
        if (n <= (int64_t)kThreads * 8)
            hipLaunchKernelGGL((select_kernel<true, true, 8>), dim3(1, nq), dim3(kThreads), 0,
                               stream, scores, nullptr, n, k, nullptr, out_ids, out_scores,
                               out_drafts, out_draft_len, spans, span_len, max_span, span_stride);
        else
            hipLaunchKernelGGL((select_kernel<true, true, kPer>), dim3(1, nq), dim3(kThreads), 0,
                               stream, scores, nullptr, n, k, nullptr, out_ids, out_scores,
                               out_drafts, out_draft_len, spans, span_len, max_span, span_stride);
        return hipGetLastError();
    }
    const size_t one = key_buffer_bytes(n, nq, k);
    uint64_t* buf[2] = {(uint64_t*)workspace, (uint64_t*)((char*)workspace + one)};
    hipLaunchKernelGGL((select_kernel<true, false, kPer>), dim3((unsigned)chunks, nq), dim3(kThreads),
                       0, stream, scores, nullptr, n, k, buf[0], nullptr, nullptr, nullptr,
                       nullptr, nullptr, nullptr, 0, 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    int64_t count = chunks * kk;
    int cur = 0;
    while ((chunks = ceil_div(count, kSelectChunk)) > 1) {
        hipLaunchKernelGGL((select_kernel<false, false, kPer>), dim3((unsigned)chunks, nq),
                           dim3(kThreads), 0, stream, nullptr, buf[cur], count, k, buf[cur ^ 1],
                           nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, 0);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        count = chunks * kk;
        cur ^= 1;
    }
    launch_final_keys(buf[cur], count, nq, k, spans, span_len, max_span, span_stride, out_ids,
                      out_scores, out_drafts, out_draft_len, stream);
    return hipGetLastError();
}

hipError_t launch_topk_keys(const uint64_t* keys, int64_t count, int nq, int k,
                            const int32_t* spans, const int32_t* span_len, int max_span,
                            int64_t span_stride, int64_t* out_ids, float* out_scores,
                            int32_t* out_drafts, int32_t* out_draft_len,
                            const int32_t* dev_count, hipStream_t stream) {
    // One block per query walks its own count.
    hipLaunchKernelGGL(select_stream_kernel, dim3(nq), dim3(kStreamThreads), 0, stream, keys,
                       count, k, dev_count, out_ids, out_scores, out_drafts, out_draft_len, spans,
                       span_len, max_span, span_stride);
    return hipGetLastError();
}

}  // namespace sense
