/*
 * A plain C99 caller of the library's C ABI (include/sense.h), linked
 * against libsense.so and the HIP runtime only: no Python, no PyTorch.  It
 * reads one retrieval + verification problem from a directory of raw files,
 * runs sense_build_index, sense_retrieve and sense_soft_gate_verify on its
 * own HIP stream with its own device buffers, and writes the results back as
 * raw files.  The GPU tests write the inputs and compare the outputs with
 * the oracle.
 *
 * Directory layout (little-endian raw arrays):
 *   params.txt     n d max_span n_queries k metric key_dtype vocab
 *                  gamma topk window tau logits_dtype
 *   keys.bin       n x d uint16 (fp16 or bf16 bits, per key_dtype)
 *   spans.bin      n x max_span int32
 *   span_len.bin   n int32
 *   queries.bin    n_queries x d float32
 *   logits.bin     (n_queries * k) x max_span x vocab, float32 or the
 *                  16-bit bits of logits_dtype
 * Outputs:
 *   ids.bin (int64), scores.bin (float32), drafts.bin, draft_len.bin,
 *   accept_len.bin, best.bin, rank.bin (int32), gate_score.bin (float32).
 *
 * Usage: sense_c_driver DIR.  Without an argument it prints this usage and
 * exits with status 2 before any HIP call.
 */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "sense.h"

#define HIP_OK(x)                                                                       \
    do {                                                                                \
        hipError_t e_ = (x);                                                            \
        if (e_ != hipSuccess) {                                                         \
            fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));              \
            return 1;                                                                   \
        }                                                                               \
    } while (0)

#define SENSE_OK_(x)                                                                    \
    do {                                                                                \
        sense_status_t s_ = (x);                                                        \
        if (s_ != SENSE_OK) {                                                           \
            fprintf(stderr, "%s failed: %s: %s\n", #x, sense_status_string(s_),         \
                    sense_last_error_message());                                        \
            return 1;                                                                   \
        }                                                                               \
    } while (0)

static char path_buf[4096];

static const char *path(const char *dir, const char *name) {
    snprintf(path_buf, sizeof path_buf, "%s/%s", dir, name);
    return path_buf;
}

/* Reads exactly `bytes` bytes of dir/name into a new host buffer. */
static void *read_all(const char *dir, const char *name, size_t bytes) {
    FILE *f = fopen(path(dir, name), "rb");
    if (!f) {
        fprintf(stderr, "cannot open %s\n", path_buf);
        return NULL;
    }
    void *p = malloc(bytes ? bytes : 1);
    const size_t got = p ? fread(p, 1, bytes, f) : 0;
    const int extra = fgetc(f);
    fclose(f);
    if (!p || got != bytes || extra != EOF) {
        fprintf(stderr, "%s: expected exactly %zu bytes\n", path_buf, bytes);
        free(p);
        return NULL;
    }
    return p;
}

static int write_all(const char *dir, const char *name, const void *p, size_t bytes) {
    FILE *f = fopen(path(dir, name), "wb");
    if (!f) {
        fprintf(stderr, "cannot create %s\n", path_buf);
        return 1;
    }
    const size_t put = fwrite(p, 1, bytes, f);
    const int closed = fclose(f);
    if (put != bytes || closed != 0) {
        fprintf(stderr, "short write to %s\n", path_buf);
        return 1;
    }
    return 0;
}

/* Copies a host array to a new device buffer. */
static int upload(void **dev, const void *host, size_t bytes) {
    HIP_OK(hipMalloc(dev, bytes ? bytes : 1));
    HIP_OK(hipMemcpy(*dev, host, bytes, hipMemcpyHostToDevice));
    return 0;
}

/* Copies a device array into a new host buffer and writes it to dir/name. */
static int download(const char *dir, const char *name, const void *dev, size_t bytes) {
    void *host = malloc(bytes ? bytes : 1);
    if (!host) return 1;
    if (hipMemcpy(host, dev, bytes, hipMemcpyDeviceToHost) != hipSuccess) {
        fprintf(stderr, "copy of %s to the host failed\n", name);
        free(host);
        return 1;
    }
    const int rc = write_all(dir, name, host, bytes);
    free(host);
    return rc;
}

int main(int argc, char **argv) {
    if (argc != 2) {
        fprintf(stderr, "usage: %s DIR (see the comment at the top of the source)\n", argv[0]);
        return 2;
    }
    const char *dir = argv[1];
    long long n, nq, k;
    int d, m, metric, key_dtype, vocab, topk, window, tau, logits_dtype;
    float gamma;
    FILE *pf = fopen(path(dir, "params.txt"), "r");
    if (!pf) {
        fprintf(stderr, "cannot open %s\n", path_buf);
        return 1;
    }
    const int fields = fscanf(pf, "%lld %d %d %lld %lld %d %d %d %f %d %d %d %d", &n, &d, &m,
                              &nq, &k, &metric, &key_dtype, &vocab, &gamma, &topk, &window, &tau,
                              &logits_dtype);
    fclose(pf);
    if (fields != 13 || n < 1 || d < 1 || m < 1 || nq < 1 || k < 1 || vocab < 1 ||
        logits_dtype < SENSE_F32 || logits_dtype > SENSE_BF16) {
        fprintf(stderr, "params.txt: expected 13 fields with positive sizes\n");
        return 1;
    }
    const long long n_cand = nq * k;
    const size_t key_bytes = (size_t)n * d * 2, span_bytes = (size_t)n * m * 4;
    const size_t q_bytes = (size_t)nq * d * 4;
    const size_t logit_bytes = (size_t)n_cand * m * vocab * (logits_dtype == SENSE_F32 ? 4 : 2);
    void *h_keys = read_all(dir, "keys.bin", key_bytes);
    void *h_spans = read_all(dir, "spans.bin", span_bytes);
    void *h_span_len = read_all(dir, "span_len.bin", (size_t)n * 4);
    void *h_queries = read_all(dir, "queries.bin", q_bytes);
    void *h_logits = read_all(dir, "logits.bin", logit_bytes);
    if (!h_keys || !h_spans || !h_span_len || !h_queries || !h_logits) return 1;

    void *keys, *spans, *span_len, *queries, *logits;
    if (upload(&keys, h_keys, key_bytes) || upload(&spans, h_spans, span_bytes) ||
        upload(&span_len, h_span_len, (size_t)n * 4) || upload(&queries, h_queries, q_bytes) ||
        upload(&logits, h_logits, logit_bytes))
        return 1;
    free(h_keys);
    free(h_spans);
    free(h_span_len);
    free(h_queries);
    free(h_logits);

    hipStream_t stream;
    HIP_OK(hipStreamCreate(&stream));

    sense_index_desc_t desc;
    memset(&desc, 0, sizeof desc);
    desc.keys = keys;
    desc.key_dtype = (sense_dtype_t)key_dtype;
    desc.n = n;
    desc.d = d;
    desc.key_stride = d;
    desc.spans = (const int32_t *)spans;
    desc.max_span = m;
    desc.span_len = (const int32_t *)span_len;
    desc.metric = (sense_metric_t)metric;
    desc.flags = 0;
    sense_index_t *index = NULL;
    SENSE_OK_(sense_build_index(&desc, stream, &index));

    /* Retrieval: ids, scores, drafts and their lengths per query. */
    size_t ws_r = 0;
    SENSE_OK_(sense_retrieve_workspace_size(index, (int32_t)nq, (int32_t)k, &ws_r));
    void *ids, *scores, *drafts, *draft_len, *workspace_r;
    HIP_OK(hipMalloc(&ids, (size_t)n_cand * 8));
    HIP_OK(hipMalloc(&scores, (size_t)n_cand * 4));
    HIP_OK(hipMalloc(&drafts, (size_t)n_cand * m * 4));
    HIP_OK(hipMalloc(&draft_len, (size_t)n_cand * 4));
    HIP_OK(hipMalloc(&workspace_r, ws_r ? ws_r : 1));
    SENSE_OK_(sense_retrieve(index, queries, SENSE_F32, (int32_t)nq, (int32_t)k,
                             (int64_t *)ids, (float *)scores, (int32_t *)drafts,
                             (int32_t *)draft_len, workspace_r, ws_r, stream));

    /* Verification of every query's k drafts (one group per query) against
     * the logits row-aligned with them. */
    sense_gate_params_t gp;
    gp.gamma = gamma;
    gp.topk = topk;
    gp.window = window;
    gp.tau = tau;
    gp.entropy_normalized = 1;
    size_t ws_v = 0;
    SENSE_OK_(sense_soft_gate_verify_workspace_size((int32_t)n_cand, m, vocab, &ws_v));
    void *accept_len, *best, *gate_score, *rank, *workspace_v;
    HIP_OK(hipMalloc(&accept_len, (size_t)n_cand * 4));
    HIP_OK(hipMalloc(&best, (size_t)nq * 4));
    HIP_OK(hipMalloc(&gate_score, (size_t)n_cand * m * 4));
    HIP_OK(hipMalloc(&rank, (size_t)n_cand * m * 4));
    HIP_OK(hipMalloc(&workspace_v, ws_v ? ws_v : 1));
    SENSE_OK_(sense_soft_gate_verify(logits, (sense_dtype_t)logits_dtype, vocab,
                                     (const int32_t *)drafts,
                                     (const int32_t *)draft_len, (int32_t)n_cand, m, vocab,
                                     (int32_t)nq, &gp, (int32_t *)accept_len, (int32_t *)best,
                                     (float *)gate_score, NULL, (int32_t *)rank, workspace_v,
                                     ws_v, stream));
    HIP_OK(hipStreamSynchronize(stream));

    if (download(dir, "ids.bin", ids, (size_t)n_cand * 8) ||
        download(dir, "scores.bin", scores, (size_t)n_cand * 4) ||
        download(dir, "drafts.bin", drafts, (size_t)n_cand * m * 4) ||
        download(dir, "draft_len.bin", draft_len, (size_t)n_cand * 4) ||
        download(dir, "accept_len.bin", accept_len, (size_t)n_cand * 4) ||
        download(dir, "best.bin", best, (size_t)nq * 4) ||
        download(dir, "gate_score.bin", gate_score, (size_t)n_cand * m * 4) ||
        download(dir, "rank.bin", rank, (size_t)n_cand * m * 4))
        return 1;

    SENSE_OK_(sense_destroy_index(index));
    void *bufs[] = {keys, spans, span_len, queries, logits, ids, scores, drafts, draft_len,
                    workspace_r, accept_len, best, gate_score, rank, workspace_v};
    for (size_t i = 0; i < sizeof bufs / sizeof bufs[0]; ++i) HIP_OK(hipFree(bufs[i]));
    HIP_OK(hipStreamDestroy(stream));
    printf("sense_c_driver: %lld queries x k=%lld over %lld x %d keys, %lld drafts verified\n",
           nq, k, n, d, n_cand);
    return 0;
}
