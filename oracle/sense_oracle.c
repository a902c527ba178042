/*
 * sense_oracle.c -- plain, slow, obviously-correct CPU reference for the
 * SENSE retrieval + soft-gated evaluation hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the oracle, not the product: only
 * the test-suite, the smoke check and the benchmark's CPU-baseline leg may
 * load it.  It shares no source, header, table or helper with the HIP library
 * and includes nothing from it.
 *
 * Every quantity is computed in IEEE double precision, following the paper's
 * definitions literally:
 *
 *   Retrieval (Sec. 3.1 Eq. 3 "retriever R", Sec. 3.2 Eq. 8 "sim",
 *   Alg. 2 "L2Norm" and "FAISS" steps):  the exact similarity of the query to
 *   every stored key (inner product, or cosine = inner product of the
 *   L2-normalised vectors), then a FULL sort of all N rows by
 *   (score descending, row index ascending) and the first k rows; the stored
 *   continuation span of each hit is gathered into the candidate batch.
 *   The paper's own retriever is an approximate (IVF-PQ) index; the exact
 *   scan is the plain definition that index approximates.
 *
 *   Verification (Sec. 3.3 Eqs. 12-18, Alg. 4 "SGE"): per candidate c and
 *   draft position j, the greedy token Y = argmax (first occurrence), the
 *   exact-match mask, softmax entropy (optionally divided by log|V|) against
 *   gamma, top-k membership of the draft token (full stable sort of the
 *   vocabulary), the padded mismatch window of width W, the final gate G,
 *   the leading run of accepted positions and the best candidate per group.
 *
 * Readings taken where the paper is silent or inconsistent (each one is also
 * listed with its reason in the design notes of the repository):
 *   - entropy is normalised by ln|V| when entropy_normalized != 0 (Alg. 4),
 *     raw nats otherwise (Eq. 14's text form);
 *   - softmax is applied to raw logits at temperature 1;
 *   - top-k ties are broken by lower vocabulary index; argmax takes the first
 *     maximum; the best candidate is the first one with the largest length;
 *   - the look-ahead window of position j is the W positions strictly after
 *     j, the draft right-padded with W mismatches (Alg. 4's Pad + Conv1D +
 *     [1:M+1] slice); B_con = (R <= tau), tau = 0 being Alg. 4's "R = 0";
 *   - positions j >= draft_len[c] are rejected and count as mismatches;
 *   - a draft id outside [0, V) matches nothing and is in no top-k set;
 *   - accept_len is the count of leading accepted positions n in [0, len];
 *     Alg. 4's L equals n - 1;
 *   - retrieval ties go to the lower row index; NaN scores sort last; a
 *     zero-norm key or query has cosine 0.
 *
 * dtype codes: 0 = float32, 1 = IEEE binary16, 2 = bfloat16.
 * All functions return 0 on success, -1 on a bad argument.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_F32 = 0, OR_F16 = 1, OR_BF16 = 2 };

/* IEEE 754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.
 * Written from the format's definition; every binary16 value is exact in
 * double. */
double oracle_decode_f16(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);               /* zero / subnormal */
    else if (e == 31)
        v = (f == 0) ? INFINITY : NAN;           /* inf / NaN */
    else
        v = ldexp((double)(1024 + f), e - 25);   /* (1 + f/1024) * 2^(e-15) */
    return sign ? -v : v;
}

/* bfloat16 is the upper half of an IEEE binary32 pattern. */
double oracle_decode_bf16(uint16_t b)
{
    uint32_t u = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double elem(const void *base, int dtype, int64_t i)
{
    switch (dtype) {
    case OR_F32: return (double)((const float *)base)[i];
    case OR_F16: return oracle_decode_f16(((const uint16_t *)base)[i]);
    default:     return oracle_decode_bf16(((const uint16_t *)base)[i]);
    }
}

static int dtype_ok(int dt) { return dt == OR_F32 || dt == OR_F16 || dt == OR_BF16; }

/* ---------------------------------------------------------------- retrieval */

/* scores[q * n + i] = sim(query q, key row i) for rows [0, n) of the block
 * given.  metric 0 = inner product, 1 = cosine.  Rows are independent, so the
 * row loop may run on several threads; each row's sum is taken in element
 * order. */
int oracle_scores(const void *keys, int key_dtype, int64_t n, int32_t d,
                  int64_t key_stride, const void *queries, int q_dtype,
                  int32_t n_queries, int metric, double *out_scores)
{
    if (!keys || !queries || !out_scores || n < 0 || d < 1 || key_stride < d ||
        n_queries < 1 || !dtype_ok(key_dtype) || !dtype_ok(q_dtype) ||
        (metric != 0 && metric != 1))
        return -1;
    for (int32_t q = 0; q < n_queries; ++q) {
        double qn2 = 0.0;
        for (int32_t t = 0; t < d; ++t) {
            double a = elem(queries, q_dtype, (int64_t)q * d + t);
            qn2 += a * a;
        }
        double qnorm = sqrt(qn2);
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < n; ++i) {
            double dot = 0.0, kn2 = 0.0;
            for (int32_t t = 0; t < d; ++t) {
                double kv = elem(keys, key_dtype, i * key_stride + t);
                double qv = elem(queries, q_dtype, (int64_t)q * d + t);
                dot += qv * kv;
                kn2 += kv * kv;
            }
            double s;
            if (metric == 0) {
                s = dot;
            } else {
                double knorm = sqrt(kn2);
                s = (knorm == 0.0 || qnorm == 0.0) ? 0.0 : dot / (qnorm * knorm);
            }
            out_scores[(int64_t)q * n + i] = s;
        }
    }
    return 0;
}

typedef struct { double s; int64_t i; } scored_row;

/* (score descending, index ascending); NaN after every number. */
static int cmp_rows(const void *pa, const void *pb)
{
    const scored_row *a = (const scored_row *)pa, *b = (const scored_row *)pb;
    int an = isnan(a->s), bn = isnan(b->s);
    if (an != bn) return an ? 1 : -1;
    if (!an) {
        if (a->s > b->s) return -1;
        if (a->s < b->s) return 1;
    }
    return (a->i < b->i) ? -1 : (a->i > b->i);
}

/* Full sort of all n scores, first k kept.  k may exceed n: the tail is
 * filled with id -1 and score NaN. */
int oracle_topk(const double *scores, int64_t n, int32_t k, int64_t *out_ids,
                double *out_scores)
{
    if (!scores || !out_ids || !out_scores || n < 0 || k < 0) return -1;
    scored_row *all = (scored_row *)malloc(sizeof(scored_row) * (size_t)(n > 0 ? n : 1));
    if (!all) return -1;
    for (int64_t i = 0; i < n; ++i) { all[i].s = scores[i]; all[i].i = i; }
    qsort(all, (size_t)n, sizeof(scored_row), cmp_rows);
    for (int32_t r = 0; r < k; ++r) {
        if (r < n) { out_ids[r] = all[r].i; out_scores[r] = all[r].s; }
        else { out_ids[r] = -1; out_scores[r] = NAN; }
    }
    free(all);
    return 0;
}

/* drafts[r][j] = spans[ids[r]][j] for j < span_len[ids[r]], else -1.
 * span_len may be NULL (every span is max_span long).  An id of -1 yields an
 * empty draft. */
int oracle_gather(const int32_t *spans, const int32_t *span_len, int32_t max_span,
                  const int64_t *ids, int32_t k, int32_t *out_drafts,
                  int32_t *out_draft_len)
{
    if (!spans || !ids || !out_drafts || !out_draft_len || max_span < 1 || k < 0)
        return -1;
    for (int32_t r = 0; r < k; ++r) {
        int64_t id = ids[r];
        int32_t len = 0;
        if (id >= 0) {
            len = span_len ? span_len[id] : max_span;
            if (len < 0) len = 0;
            if (len > max_span) len = max_span;
        }
        for (int32_t j = 0; j < max_span; ++j)
            out_drafts[(int64_t)r * max_span + j] =
                (j < len) ? spans[id * max_span + j] : -1;
        out_draft_len[r] = len;
    }
    return 0;
}

/* ------------------------------------------------------------- verification */

typedef struct { double x; int32_t v; } vocab_entry;

static int cmp_vocab(const void *pa, const void *pb)
{
    const vocab_entry *a = (const vocab_entry *)pa, *b = (const vocab_entry *)pb;
    if (a->x > b->x) return -1;
    if (a->x < b->x) return 1;
    return (a->v < b->v) ? -1 : (a->v > b->v);
}

/* Statistics of one logit row x[0..V) judged against draft token tok:
 *   argmax (first occurrence), entropy of softmax(x) in nats,
 *   rank = position of tok in the stable sort by (x desc, v asc) (V if tok is
 *   outside [0, V)).  tok is in the top-k set iff rank < k. */
int oracle_row_stats(const void *row, int dtype, int32_t vocab, int32_t tok,
                     int32_t *out_argmax, double *out_entropy, int32_t *out_rank)
{
    if (!row || vocab < 1 || !dtype_ok(dtype)) return -1;
    vocab_entry *e = (vocab_entry *)malloc(sizeof(vocab_entry) * (size_t)vocab);
    if (!e) return -1;
    int32_t y = 0;
    double m = elem(row, dtype, 0);
    for (int32_t v = 0; v < vocab; ++v) {
        e[v].x = elem(row, dtype, v);
        e[v].v = v;
        if (e[v].x > m) { m = e[v].x; y = v; }
    }
    /* softmax p_v = exp(x_v - m) / sum_u exp(x_u - m); entropy -sum p ln p.
     * With m = +inf the weights exp(x_v - m) are undefined (+inf - +inf), so
     * the entropy is too: NaN (never above gamma). */
    double ent = 0.0;
    if (isinf(m) && m > 0) {
        ent = NAN;
    } else {
        double z = 0.0;
        for (int32_t v = 0; v < vocab; ++v) z += exp(e[v].x - m);
        for (int32_t v = 0; v < vocab; ++v) {
            double p = exp(e[v].x - m) / z;
            if (p > 0.0) ent -= p * log(p);
        }
    }
    int32_t rank = vocab;
    if (tok >= 0 && tok < vocab) {
        qsort(e, (size_t)vocab, sizeof(vocab_entry), cmp_vocab);
        for (int32_t r = 0; r < vocab; ++r)
            if (e[r].v == tok) { rank = r; break; }
    }
    free(e);
    if (out_argmax) *out_argmax = y;
    if (out_entropy) *out_entropy = ent;
    if (out_rank) *out_rank = rank;
    return 0;
}

/* Soft-gated evaluation of n_cand drafts (row-major n_cand x max_len) against
 * the aligned logits: row (c, j) starts at logits + (c*max_len + j)*row_stride
 * and predicts drafts[c][j].  draft_len may be NULL (all max_len).  Rows at
 * j >= draft_len[c] are never read.
 *
 * Outputs (NULL allowed for the optional ones):
 *   accept_len[c]  leading accepted count n_c
 *   best[g]        index within group g of its first candidate of largest n
 *   gate_score[c*max_len + j]  the value compared with gamma (0 beyond len)
 *   masks[c*max_len + j]       em | ent<<1 | topk<<2 | con<<3 | G<<4
 *   argmax / rank  per position (-1 / V beyond len) */
int oracle_soft_gate_verify(const void *logits, int logits_dtype, int64_t row_stride,
                            const int32_t *drafts, const int32_t *draft_len,
                            int32_t n_cand, int32_t max_len, int32_t vocab,
                            int32_t n_groups, double gamma, int32_t topk,
                            int32_t window, int32_t tau, int32_t entropy_normalized,
                            int32_t *out_accept_len, int32_t *out_best,
                            double *out_gate_score, uint8_t *out_masks,
                            int32_t *out_argmax, int32_t *out_rank)
{
    if (n_cand < 0 || max_len < 1 || vocab < 1 || row_stride < vocab ||
        topk < 1 || window < 0 || tau < 0 || !dtype_ok(logits_dtype) ||
        (n_cand > 0 && (!logits || !drafts || !out_accept_len)))
        return -1;
    if (n_cand > 0 && (n_groups < 1 || n_cand % n_groups != 0)) return -1;
    const int64_t npos = (int64_t)n_cand * max_len;
    uint8_t *em = (uint8_t *)calloc((size_t)(npos > 0 ? npos : 1), 1);
    uint8_t *ent = (uint8_t *)calloc((size_t)(npos > 0 ? npos : 1), 1);
    uint8_t *tk = (uint8_t *)calloc((size_t)(npos > 0 ? npos : 1), 1);
    double *gs = (double *)calloc((size_t)(npos > 0 ? npos : 1), sizeof(double));
    int32_t *am = (int32_t *)malloc(sizeof(int32_t) * (size_t)(npos > 0 ? npos : 1));
    int32_t *rk = (int32_t *)malloc(sizeof(int32_t) * (size_t)(npos > 0 ? npos : 1));
    int32_t *lens = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_cand > 0 ? n_cand : 1));
    if (!em || !ent || !tk || !gs || !am || !rk || !lens) {
        free(em); free(ent); free(tk); free(gs); free(am); free(rk); free(lens);
        return -1;
    }
    const double log_v = log((double)vocab);
    for (int32_t c = 0; c < n_cand; ++c) {
        int32_t len = draft_len ? draft_len[c] : max_len;
        if (len < 0) len = 0;
        if (len > max_len) len = max_len;
        lens[c] = len;
    }

    /* Per-position masks: exact match, entropy gate, top-k membership. */
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < npos; ++p) {
        int32_t c = (int32_t)(p / max_len), j = (int32_t)(p % max_len);
        am[p] = -1;
        rk[p] = vocab;
        if (j >= lens[c]) continue;              /* beyond the draft: rejected */
        int32_t tok = drafts[p];
        int32_t y, r;
        double e;
        const char *row = (const char *)logits +
                          (size_t)p * (size_t)row_stride *
                              (logits_dtype == OR_F32 ? 4 : 2);
        if (oracle_row_stats(row, logits_dtype, vocab, tok, &y, &e, &r)) { err = 1; continue; }
        /* |V| = 1: E = 0 and E / ln|V| is 0/0; it is read as 0 */
        double g = entropy_normalized ? (vocab > 1 ? e / log_v : 0.0) : e;
        am[p] = y;
        rk[p] = r;
        em[p] = (tok == y);                      /* Y = argmax; B_em = I(D = Y) */
        ent[p] = (g > gamma);                    /* strict */
        tk[p] = (r < vocab) && (r < topk);       /* D in TopK(P, k): a vocabulary index */
        gs[p] = g;
    }
    if (err) {
        free(em); free(ent); free(tk); free(gs); free(am); free(rk); free(lens);
        return -1;
    }

    /* Per candidate: padded mismatch window, gate, leading accepted run. */
    int32_t padded_len = max_len + window;
    uint8_t *bbar = (uint8_t *)malloc((size_t)padded_len);
    for (int32_t c = 0; c < n_cand; ++c) {
        /* B-bar = Pad(1 - B_em, (0, W), value 1) */
        for (int32_t j = 0; j < padded_len; ++j)
            bbar[j] = (j < max_len) ? (uint8_t)(1 - em[(int64_t)c * max_len + j]) : 1;
        int32_t n = 0, still = 1;
        for (int32_t j = 0; j < max_len; ++j) {
            int64_t p = (int64_t)c * max_len + j;
            /* R[j] = sum over the W positions after j */
            int32_t r = 0;
            for (int32_t u = 1; u <= window; ++u) r += bbar[j + u];
            int con = (r <= tau);
            int g = (j < lens[c]) &&
                    (em[p] || (ent[p] && (tk[p] || con)));
            if (still && g) ++n; else still = 0;   /* sum of cumprod(G) */
            if (out_masks)
                out_masks[p] = (uint8_t)(em[p] | (ent[p] << 1) | (tk[p] << 2) |
                                         (con << 3) | (g << 4));
            if (out_gate_score) out_gate_score[p] = gs[p];
            if (out_argmax) out_argmax[p] = am[p];
            if (out_rank) out_rank[p] = rk[p];
        }
        out_accept_len[c] = n;
    }
    free(bbar);

    /* Best candidate of each group: first maximiser of n. */
    if (out_best && n_cand > 0) {
        int32_t gsz = n_cand / n_groups;
        for (int32_t g = 0; g < n_groups; ++g) {
            int32_t b = 0;
            for (int32_t i = 1; i < gsz; ++i)
                if (out_accept_len[g * gsz + i] > out_accept_len[g * gsz + b]) b = i;
            out_best[g] = b;
        }
    }
    free(em); free(ent); free(tk); free(gs); free(am); free(rk); free(lens);
    return 0;
}

/* ------------------------------------------------------ candidate selection */

typedef struct { double s; int32_t i; } ranked_cand;

/* (composite score descending, position in D_all ascending); NaN last. */
static int cmp_cand(const void *pa, const void *pb)
{
    const ranked_cand *a = (const ranked_cand *)pa, *b = (const ranked_cand *)pb;
    int an = isnan(a->s), bn = isnan(b->s);
    if (an != bn) return an ? 1 : -1;
    if (!an) {
        if (a->s > b->s) return -1;
        if (a->s < b->s) return 1;
    }
    return (a->i < b->i) ? -1 : (a->i > b->i);
}

/* Candidate selection of one query (Sec. 3.2 Eq. 8; Alg. 2 hybrid retrieval,
 * composite score, Top-N and anchor override), literally:
 *   D_all = static hits (n_s) followed by dynamic hits (n_d);
 *   s     = [scores_s ; scores_d + delta];
 *   S_i   = alpha * I(D_all[i][0] == anchor) + beta * s_i   (a draft of
 *           length 0 has no first token: I = 0);
 *   D     = the top_n rows of D_all by (S desc, i asc), full sort;
 *   if anchor_override: D[0][0] = anchor and D[top_n-1][0] = anchor (a row
 *           of length 0 becomes length 1).
 * Drafts are n x max_len int32 padded with -1, lengths n.  Outputs
 * top_n x max_len drafts, top_n lengths, the position of each selected row in
 * D_all (source) and its composite score.  top_n <= n_s + n_d.
 * f32 != 0 takes the composite score in binary32 (see the loop) so that an
 * implementation computing in binary32 can be compared order-exactly; the
 * order is still a full sort by the same rule. */
int oracle_select_candidates(const double *scores_s, const int32_t *drafts_s,
                             const int32_t *len_s, int32_t n_s,
                             const double *scores_d, const int32_t *drafts_d,
                             const int32_t *len_d, int32_t n_d, int32_t anchor,
                             int32_t max_len, int32_t top_n, double alpha, double beta,
                             double delta, int32_t anchor_override, int32_t f32,
                             int32_t *out_drafts, int32_t *out_len, int32_t *out_source,
                             double *out_score)
{
    int32_t n_all = n_s + n_d;
    if (n_s < 0 || n_d < 0 || max_len < 1 || top_n < 1 || top_n > n_all ||
        !out_drafts || !out_len || (n_s > 0 && (!scores_s || !drafts_s)) ||
        (n_d > 0 && (!scores_d || !drafts_d)))
        return -1;
    ranked_cand *c = (ranked_cand *)malloc(sizeof(ranked_cand) * (size_t)n_all);
    if (!c) return -1;
    for (int32_t i = 0; i < n_all; ++i) {
        int dyn = i >= n_s;
        int32_t r = dyn ? i - n_s : i;
        const int32_t *row = (dyn ? drafts_d : drafts_s) + (int64_t)r * max_len;
        int32_t len = dyn ? (len_d ? len_d[r] : max_len) : (len_s ? len_s[r] : max_len);
        int match = len > 0 && row[0] == anchor;
        if (f32) {
            /* The same formula taken in binary32, rounding each step:
             * s = fl(s_d + delta) for dynamic hits, S = fl(beta * s + alpha * I)
             * as one fused multiply-add (C99 fmaf rounds once). */
            float sf = dyn ? (float)scores_d[r] + (float)delta : (float)scores_s[r];
            c[i].s = (double)fmaf((float)beta, sf, match ? (float)alpha : 0.0f);
        } else {
            double s = dyn ? scores_d[r] + delta : scores_s[r];
            c[i].s = alpha * (match ? 1.0 : 0.0) + beta * s;
        }
        c[i].i = i;
    }
    qsort(c, (size_t)n_all, sizeof(ranked_cand), cmp_cand);
    for (int32_t r = 0; r < top_n; ++r) {
        int32_t i = c[r].i;
        int dyn = i >= n_s;
        int32_t src = dyn ? i - n_s : i;
        const int32_t *row = (dyn ? drafts_d : drafts_s) + (int64_t)src * max_len;
        int32_t len = dyn ? (len_d ? len_d[src] : max_len) : (len_s ? len_s[src] : max_len);
        if (len < 0) len = 0;
        if (len > max_len) len = max_len;
        for (int32_t j = 0; j < max_len; ++j)
            out_drafts[(int64_t)r * max_len + j] = j < len ? row[j] : -1;
        out_len[r] = len;
        if (out_source) out_source[r] = i;
        if (out_score) out_score[r] = c[r].s;
    }
    if (anchor_override) {
        int32_t ends[2] = {0, top_n - 1};
        for (int e = 0; e < 2; ++e) {
            int32_t r = ends[e];
            out_drafts[(int64_t)r * max_len] = anchor;
            if (out_len[r] < 1) out_len[r] = 1;
        }
    }
    free(c);
    return 0;
}

/* ---------------------------------------------------------------- projection */

/* Query / key construction of Alg. 2 (k = L2Norm(PCA(h))) and the datastore
 * projection Z of Sec. 3.2 Eq. 6 with the PCA of the implementation details:
 *   out[i][o] = sum_t (x[i][t] - mean[t]) * basis[o][t]   (mean NULL = 0)
 * then, if normalize, out[i] /= ||out[i]|| (a zero row stays zero).
 * x is n x d_in of x_dtype with row stride x_stride; basis is d_out x d_in
 * fp64 (the principal directions as rows); mean d_in fp64.  Sums in element
 * order, in double precision. */
int oracle_project(const void *x, int x_dtype, int64_t n, int32_t d_in, int64_t x_stride,
                   const double *mean, const double *basis, int32_t d_out, int32_t normalize,
                   double *out)
{
    if (!x || !basis || !out || !dtype_ok(x_dtype) || n < 0 || d_in < 1 || d_out < 1 ||
        x_stride < d_in)
        return -1;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double *row = out + i * d_out;
        for (int32_t o = 0; o < d_out; ++o) {
            double s = 0.0;
            for (int32_t t = 0; t < d_in; ++t) {
                double c = elem(x, x_dtype, i * x_stride + t) - (mean ? mean[t] : 0.0);
                s += c * basis[(int64_t)o * d_in + t];
            }
            row[o] = s;
        }
        if (normalize) {
            double nn = 0.0;
            for (int32_t o = 0; o < d_out; ++o) nn += row[o] * row[o];
            if (nn > 0.0) {
                double inv = 1.0 / sqrt(nn);
                for (int32_t o = 0; o < d_out; ++o) row[o] *= inv;
            }
        }
    }
    return 0;
}

/* ---------------------------------------------------------------- IVF / IVF-PQ */

/* Similarity of a key row to a double vector under the index metric:
 * inner product, or cosine (0 when either norm is 0). */
static double sim_row(const void *keys, int key_dtype, int64_t off, int32_t d, const double *v,
                      int metric)
{
    double dot = 0.0, kn = 0.0, vn = 0.0;
    for (int32_t t = 0; t < d; ++t) {
        double x = elem(keys, key_dtype, off + t);
        dot += x * v[t];
        kn += x * x;
        vn += v[t] * v[t];
    }
    if (metric == 0) return dot;
    return (kn == 0.0 || vn == 0.0) ? 0.0 : dot / (sqrt(kn) * sqrt(vn));
}

/* Coarse quantizer of the inverted file (the FAISS IVF index of the
 * implementation details): each key joins the list of the centroid it is most
 * similar to under the index metric (ties: lower list id). */
int oracle_ivf_assign(const void *keys, int key_dtype, int64_t n, int32_t d, int64_t key_stride,
                      const double *centroids, int32_t nlist, int metric, int32_t *out_list,
                      double *out_score)
{
    if (!keys || !centroids || !out_list || nlist < 1 || d < 1 || key_stride < d ||
        !dtype_ok(key_dtype))
        return -1;
    /* The same sums as sim_row, term for term and in the same order, with
     * each centroid's squared norm formed once and each key decoded once
     * (every similarity is the value sim_row gives). */
    double *vn = malloc((size_t)nlist * sizeof(double));
    if (!vn) return -1;
    for (int32_t l = 0; l < nlist; ++l) {
        const double *v = centroids + (int64_t)l * d;
        double s = 0.0;
        for (int32_t t = 0; t < d; ++t) s += v[t] * v[t];
        vn[l] = s;
    }
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double *x = malloc((size_t)d * sizeof(double));
        double kn = 0.0;
        for (int32_t t = 0; t < d; ++t) {
            x[t] = elem(keys, key_dtype, i * key_stride + t);
            kn += x[t] * x[t];
        }
        int32_t best = 0;
        double bs = -INFINITY;
        for (int32_t l = 0; l < nlist; ++l) {
            const double *v = centroids + (int64_t)l * d;
            double dot = 0.0;
            for (int32_t t = 0; t < d; ++t) dot += x[t] * v[t];
            double s = dot;
            if (metric != 0)
                s = (kn == 0.0 || vn[l] == 0.0) ? 0.0 : dot / (sqrt(kn) * sqrt(vn[l]));
            if (s > bs) { bs = s; best = l; }
        }
        out_list[i] = best;
        if (out_score) out_score[i] = bs;
        free(x);
    }
    free(vn);
    return 0;
}

/* Product quantizer of the residuals (IVF-PQ, m sub-quantizers of
 * dsub = d / m dimensions, ksub centroids each): code j of key i is the
 * codebook entry nearest (squared L2, ties: lower entry) to the j-th slice of
 * r_i = key_i - centroid[list_i].  codebooks is m x ksub x dsub. */
int oracle_pq_encode(const void *keys, int key_dtype, int64_t n, int32_t d, int64_t key_stride,
                     const double *centroids, const int32_t *list_ids, const double *codebooks,
                     int32_t m, int32_t ksub, uint8_t *out_codes)
{
    if (!keys || !centroids || !list_ids || !codebooks || !out_codes || m < 1 || d % m != 0 ||
        ksub < 1 || ksub > 256 || !dtype_ok(key_dtype))
        return -1;
    int32_t dsub = d / m;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const double *c = centroids + (int64_t)list_ids[i] * d;
        for (int32_t j = 0; j < m; ++j) {
            int32_t best = 0;
            double bd = INFINITY;
            for (int32_t e = 0; e < ksub; ++e) {
                const double *cb = codebooks + ((int64_t)j * ksub + e) * dsub;
                double dist = 0.0;
                for (int32_t t = 0; t < dsub; ++t) {
                    double r = elem(keys, key_dtype, i * key_stride + j * dsub + t) - c[j * dsub + t];
                    double df = r - cb[t];
                    dist += df * df;
                }
                if (dist < bd) { bd = dist; best = e; }
            }
            out_codes[i * m + j] = (uint8_t)best;
        }
    }
    return 0;
}

typedef struct { double s; int32_t i; } scored_list;

static int cmp_lists(const void *pa, const void *pb)
{
    const scored_list *a = (const scored_list *)pa, *b = (const scored_list *)pb;
    int an = isnan(a->s), bn = isnan(b->s);
    if (an != bn) return an ? 1 : -1;
    if (!an) {
        if (a->s > b->s) return -1;
        if (a->s < b->s) return 1;
    }
    return (a->i < b->i) ? -1 : (a->i > b->i);
}

/* IVF search of one query (exact re-ranking inside the probed lists for
 * IVF-Flat, asymmetric distance computation for IVF-PQ):
 *   coarse[l] = sim(q, centroid l) under the index metric;
 *   probe     = the nprobe lists with the largest coarse score (full sort,
 *               ties: lower list id);
 *   candidates = every key whose list is probed, scored by
 *     IVF-Flat: the exact similarity of the key (as oracle_scores), or
 *     IVF-PQ (codes != NULL): u . (centroid[list] + reconstruction), with
 *       u = q (IP) or q / ||q|| (cosine) and the reconstruction the
 *       concatenated codebook entries of the key's codes;
 *   result    = the k best candidates, full sort (score desc, row asc); k may
 *               exceed the candidate count: the tail is id -1, score NaN.
 * query is d doubles. */
int oracle_ivf_search(const double *query, int32_t d, const double *centroids, int32_t nlist,
                      int metric, int32_t nprobe, const int32_t *list_ids, int64_t n,
                      const void *keys, int key_dtype, int64_t key_stride,
                      const uint8_t *codes, const double *codebooks, int32_t m, int32_t ksub,
                      int32_t k, int32_t *out_probe, double *out_coarse, int64_t *out_ids,
                      double *out_scores)
{
    if (!query || !centroids || !list_ids || nlist < 1 || nprobe < 1 || nprobe > nlist ||
        k < 1 || (!codes && !keys) || (codes && (!codebooks || m < 1 || d % m != 0)))
        return -1;
    double qn = 0.0;
    for (int32_t t = 0; t < d; ++t) qn += query[t] * query[t];
    qn = sqrt(qn);
    scored_list *ls = (scored_list *)malloc(sizeof(scored_list) * (size_t)nlist);
    if (!ls) return -1;
    for (int32_t l = 0; l < nlist; ++l) {
        const double *c = centroids + (int64_t)l * d;
        double dot = 0.0, cn = 0.0;
        for (int32_t t = 0; t < d; ++t) { dot += query[t] * c[t]; cn += c[t] * c[t]; }
        cn = sqrt(cn);
        ls[l].s = metric == 0 ? dot : ((cn == 0.0 || qn == 0.0) ? 0.0 : dot / (qn * cn));
        ls[l].i = l;
        if (out_coarse) out_coarse[l] = ls[l].s;
    }
    qsort(ls, (size_t)nlist, sizeof(scored_list), cmp_lists);
    char *probed = (char *)calloc((size_t)nlist, 1);
    if (!probed) { free(ls); return -1; }
    for (int32_t p = 0; p < nprobe; ++p) {
        probed[ls[p].i] = 1;
        if (out_probe) out_probe[p] = ls[p].i;
    }
    int64_t cnt = 0;
    for (int64_t i = 0; i < n; ++i) cnt += probed[list_ids[i]];
    scored_row *cand = (scored_row *)malloc(sizeof(scored_row) * (size_t)(cnt > 0 ? cnt : 1));
    if (!cand) { free(ls); free(probed); return -1; }
    int32_t dsub = codes ? d / m : 0;
    double u_scale = (metric == 0 || qn == 0.0) ? 1.0 : 1.0 / qn;
    int64_t c = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (!probed[list_ids[i]]) continue;
        double s;
        if (!codes) {
            s = sim_row(keys, key_dtype, i * key_stride, d, query, metric);
        } else {
            const double *cen = centroids + (int64_t)list_ids[i] * d;
            s = 0.0;
            for (int32_t j = 0; j < m; ++j) {
                const double *cb = codebooks + ((int64_t)j * ksub + codes[i * m + j]) * dsub;
                for (int32_t t = 0; t < dsub; ++t)
                    s += (query[j * dsub + t] * u_scale) * (cen[j * dsub + t] + cb[t]);
            }
        }
        cand[c].s = s;
        cand[c].i = i;
        ++c;
    }
    qsort(cand, (size_t)cnt, sizeof(scored_row), cmp_rows);
    for (int32_t r = 0; r < k; ++r) {
        out_ids[r] = r < cnt ? cand[r].i : -1;
        out_scores[r] = r < cnt ? cand[r].s : NAN;
    }
    free(ls); free(probed); free(cand);
    return 0;
}
