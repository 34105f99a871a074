/* Host-only driver of the oracle, for builds with the address and
 * undefined-behaviour sanitizers (tests/test_host_sanitizers.py).
 *
 *   oracle_driver LIST ASR K OUT
 *
 * LIST: the binary n-gram list of build_driver.cpp.  ASR: int64 B, int64 T,
 * then float [B, T, V + 1].  Writes to OUT, in order: the advance of every
 * state (float scores [S, V], int32 next [S, V]), a plain and a CTC decode of
 * ASR from state 0 (int32 labels and states [B, T] each; an AED decode from
 * the start state too when the list carries <s> and </s>), the top-k of frame
 * 0 of each utterance at the first B states (int32 tokens, float scores, int32
 * next, [B, K] each) and, with <s> and </s>, the final weights of every state. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct oracle_model oracle_model;
int oracle_create(int32_t V, int32_t N, int64_t M, const int32_t *order, const int32_t *tokens,
                  const float *logprob, const float *backoff, float unk_logprob, int flags, oracle_model **out);
void oracle_free(oracle_model *m);
int64_t oracle_num_states(const oracle_model *m);
int64_t oracle_start_state(const oracle_model *m);
int oracle_advance(const oracle_model *m, const int32_t *states, int64_t B, float *scores32, double *scores64,
                   int32_t *next, int nthreads);
int oracle_decode(const oracle_model *m, const float *asr, int64_t B, int64_t T, int64_t ld, int mode, float lambda,
                  const int32_t *starts, const int32_t *lengths, const int32_t *prev0, int32_t *labels,
                  int32_t *states_out, int nthreads);
int oracle_fused_topk(const oracle_model *m, const float *asr, int64_t B, int64_t ld, float lambda, int k,
                      const int32_t *states, int32_t *tokens, float *scores, int32_t *next);
int oracle_final(const oracle_model *m, const int32_t *states, int64_t B, float *out);
int oracle_repair(int32_t V, int32_t N, int64_t M, const int32_t *order, const int32_t *tokens,
                  const float *logprob, const float *backoff, float unk_logprob, int flags, int64_t *M_out,
                  int32_t **order_out, int32_t **tokens_out, float **W_out, float **B_out);
void oracle_free_buffer(void *p);

static void *read_all(const char *path, size_t *n) {
    FILE *f = fopen(path, "rb");
    if (!f) return NULL;
    fseek(f, 0, SEEK_END);
    long len = ftell(f);
    fseek(f, 0, SEEK_SET);
    void *p = malloc(len > 0 ? (size_t)len : 1);
    *n = fread(p, 1, (size_t)len, f);
    fclose(f);
    return p;
}

static void put(FILE *f, const void *p, size_t bytes) { fwrite(p, 1, bytes, f); }

/* oracle_driver repair LIST OUT: the repaired list (int64 M, then order, tokens, W, B). */
static int repair_main(const char *list_path, const char *out_path) {
    size_t n = 0;
    char *buf = (char *)read_all(list_path, &n);
    if (!buf || n < 24) return 2;
    int32_t V = *(int32_t *)buf, N = *(int32_t *)(buf + 4);
    int64_t M = *(int64_t *)(buf + 8);
    float unk = *(float *)(buf + 16);
    uint32_t flags = *(uint32_t *)(buf + 20);
    const int32_t *order = (const int32_t *)(buf + 24);
    const int32_t *tokens = order + M;
    const float *W = (const float *)(tokens + M * N);
    const float *Bk = W + M;
    int64_t M2 = 0;
    int32_t *o2 = NULL, *t2 = NULL;
    float *w2 = NULL, *b2 = NULL;
    int rc = oracle_repair(V, N, M, order, tokens, W, Bk, unk, (int)(flags & 1u), &M2, &o2, &t2, &w2, &b2);
    if (rc) { fprintf(stderr, "oracle_repair rc %d\n", rc); free(buf); return 3; }
    FILE *out = fopen(out_path, "wb");
    put(out, &M2, sizeof M2);
    put(out, o2, sizeof(int32_t) * (size_t)M2);
    put(out, t2, sizeof(int32_t) * (size_t)(M2 * N));
    put(out, w2, sizeof(float) * (size_t)M2);
    put(out, b2, sizeof(float) * (size_t)M2);
    fclose(out);
    oracle_free_buffer(o2); oracle_free_buffer(t2); oracle_free_buffer(w2); oracle_free_buffer(b2);
    free(buf);
    printf("rc 0 rows %lld\n", (long long)M2);
    return 0;
}

int main(int argc, char **argv) {
    if (argc == 4 && argv[1][0] == 'r') return repair_main(argv[2], argv[3]);
    if (argc != 5) { fprintf(stderr, "usage: oracle_driver LIST ASR K OUT | repair LIST OUT\n"); return 2; }
    size_t n = 0, na = 0;
    char *buf = (char *)read_all(argv[1], &n);
    char *abuf = (char *)read_all(argv[2], &na);
    if (!buf || !abuf || n < 24 || na < 16) { fprintf(stderr, "cannot read inputs\n"); return 2; }
    int32_t V = *(int32_t *)buf, N = *(int32_t *)(buf + 4);
    int64_t M = *(int64_t *)(buf + 8);
    float unk = *(float *)(buf + 16);
    uint32_t flags = *(uint32_t *)(buf + 20);
    const int32_t *order = (const int32_t *)(buf + 24);
    const int32_t *tokens = order + M;
    const float *W = (const float *)(tokens + M * N);
    const float *Bk = W + M;
    int64_t B = *(int64_t *)abuf, T = *(int64_t *)(abuf + 8);
    const float *asr = (const float *)(abuf + 16);
    int K = atoi(argv[3]);
    oracle_model *m = NULL;
    int rc = oracle_create(V, N, M, order, tokens, W, Bk, unk, (int)(flags & 1u), &m);
    if (rc) { fprintf(stderr, "oracle_create rc %d\n", rc); return 3; }
    const int64_t S = oracle_num_states(m);
    const int32_t start = (int32_t)oracle_start_state(m);
    FILE *out = fopen(argv[4], "wb");
    int32_t *st = (int32_t *)malloc(sizeof(int32_t) * (size_t)S);
    for (int64_t s = 0; s < S; ++s) st[s] = (int32_t)s;
    float *sc = (float *)malloc(sizeof(float) * (size_t)(S * V));
    int32_t *nx = (int32_t *)malloc(sizeof(int32_t) * (size_t)(S * V));
    rc = oracle_advance(m, st, S, sc, NULL, nx, 4);
    put(out, sc, sizeof(float) * (size_t)(S * V));
    put(out, nx, sizeof(int32_t) * (size_t)(S * V));
    int32_t *lab = (int32_t *)malloc(sizeof(int32_t) * (size_t)(B * T));
    int32_t *lst = (int32_t *)malloc(sizeof(int32_t) * (size_t)(B * T));
    int32_t *starts = (int32_t *)malloc(sizeof(int32_t) * (size_t)B);
    for (int mode = 0; mode <= 3 && !rc; ++mode) {
        if (mode == 2 || (mode == 3 && !(flags & 1u))) continue;
        for (int64_t b = 0; b < B; ++b) starts[b] = mode == 3 ? start : 0;
        rc = oracle_decode(m, asr, B, T, V + 1, mode, 0.5f, starts, NULL, NULL, lab, lst, 3);
        put(out, lab, sizeof(int32_t) * (size_t)(B * T));
        put(out, lst, sizeof(int32_t) * (size_t)(B * T));
    }
    if (!rc) {
        int32_t *tt = (int32_t *)malloc(sizeof(int32_t) * (size_t)(B * K));
        float *ts = (float *)malloc(sizeof(float) * (size_t)(B * K));
        int32_t *tn = (int32_t *)malloc(sizeof(int32_t) * (size_t)(B * K));
        for (int64_t b = 0; b < B; ++b) starts[b] = (int32_t)(b % S);
        rc = oracle_fused_topk(m, asr, B, T * (V + 1), 0.7f, K, starts, tt, ts, tn);
        put(out, tt, sizeof(int32_t) * (size_t)(B * K));
        put(out, ts, sizeof(float) * (size_t)(B * K));
        put(out, tn, sizeof(int32_t) * (size_t)(B * K));
        free(tt); free(ts); free(tn);
    }
    if (!rc && (flags & 1u)) {
        rc = oracle_final(m, st, S, sc);
        put(out, sc, sizeof(float) * (size_t)S);
    }
    fclose(out);
    printf("rc %d states %lld\n", rc, (long long)S);
    free(st); free(sc); free(nx); free(lab); free(lst); free(starts);
    oracle_free(m);
    free(buf); free(abuf);
    return rc ? 4 : 0;
}
