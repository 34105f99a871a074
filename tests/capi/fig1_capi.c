/* A C consumer of the library's ABI (include/ngpu_lm.h) with no Python and no
 * torch: HIP runtime calls for device memory, the library for everything else.
 * Used by tests/test_capi.py on the worked example of Section 2.1 (Figure 1).
 *
 *   fig1_capi LIST
 *
 * LIST: int32 V, int32 N, int64 M, float unk, uint32 flags, int32 order[M],
 * int32 tokens[M * N], float logprob[M], float backoff[M].
 *
 * Prints "state S v V score X next N" for every state and token (advance),
 * then "step T token V state S" for greedy plain-fusion steps at lambda = 0
 * that follow the sentence given on stdin (one token id per line), then
 * "error CODE" for one deliberately invalid call, then "ok". */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <hip/hip_runtime_api.h>

#include "ngpu_lm.h"

#define CHECK_HIP(x)                                                              \
    do {                                                                          \
        hipError_t e_ = (x);                                                      \
        if (e_ != hipSuccess) {                                                   \
            fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));              \
            return 3;                                                             \
        }                                                                         \
    } while (0)
#define CHECK_LM(x)                                                               \
    do {                                                                          \
        int r_ = (x);                                                             \
        if (r_ != NGPU_OK) {                                                      \
            fprintf(stderr, "%s: %d %s\n", #x, r_, ngpu_lm_last_error());        \
            return 4;                                                             \
        }                                                                         \
    } while (0)

int main(int argc, char **argv) {
    if (argc != 2) {
        fprintf(stderr, "usage: fig1_capi LIST < sentence\n");
        return 2;
    }
    FILE *f = fopen(argv[1], "rb");
    if (!f) return 2;
    int32_t hdr[2];
    int64_t M;
    float unk;
    uint32_t flags;
    if (fread(hdr, 4, 2, f) != 2 || fread(&M, 8, 1, f) != 1 || fread(&unk, 4, 1, f) != 1 ||
        fread(&flags, 4, 1, f) != 1 || M < 1 || hdr[1] < 1 || hdr[1] > NGPU_LM_MAX_ORDER)
        return 2;
    const int32_t V = hdr[0], N = hdr[1];
    int32_t *order = malloc(sizeof(int32_t) * (size_t)M);
    int32_t *tokens = malloc(sizeof(int32_t) * (size_t)(M * N));
    float *W = malloc(sizeof(float) * (size_t)M), *B = malloc(sizeof(float) * (size_t)M);
    if (fread(order, 4, (size_t)M, f) != (size_t)M || fread(tokens, 4, (size_t)(M * N), f) != (size_t)(M * N) ||
        fread(W, 4, (size_t)M, f) != (size_t)M || fread(B, 4, (size_t)M, f) != (size_t)M)
        return 2;
    fclose(f);

    ngpu_ngram_list list = {M, N, order, tokens, W, B};
    ngpu_lm *lm = NULL;
    CHECK_LM(ngpu_lm_build(&list, V, unk, flags, &lm));
    ngpu_lm_info_t info;
    CHECK_LM(ngpu_lm_info(lm, &info));
    const int64_t S = info.num_states;

    hipStream_t stream;
    CHECK_HIP(hipStreamCreate(&stream));
    void *img = NULL;
    const size_t bytes = ngpu_lm_device_bytes(lm);
    CHECK_HIP(hipMalloc(&img, bytes));   /* hipMalloc returns 256-byte aligned memory */
    CHECK_LM(ngpu_lm_upload(lm, img, bytes, stream));

    /* advance: every state */
    int32_t *h_states = malloc(sizeof(int32_t) * (size_t)S);
    for (int64_t s = 0; s < S; ++s) h_states[s] = (int32_t)s;
    int32_t *d_states, *d_next;
    float *d_scores;
    CHECK_HIP(hipMalloc((void **)&d_states, sizeof(int32_t) * (size_t)S));
    CHECK_HIP(hipMalloc((void **)&d_scores, sizeof(float) * (size_t)(S * V)));
    CHECK_HIP(hipMalloc((void **)&d_next, sizeof(int32_t) * (size_t)(S * V)));
    CHECK_HIP(hipMemcpyAsync(d_states, h_states, sizeof(int32_t) * (size_t)S, hipMemcpyHostToDevice, stream));
    CHECK_LM(ngpu_lm_advance(lm, d_states, S, d_scores, d_next, stream));
    float *h_scores = malloc(sizeof(float) * (size_t)(S * V));
    int32_t *h_next = malloc(sizeof(int32_t) * (size_t)(S * V));
    CHECK_HIP(hipMemcpyAsync(h_scores, d_scores, sizeof(float) * (size_t)(S * V), hipMemcpyDeviceToHost, stream));
    CHECK_HIP(hipMemcpyAsync(h_next, d_next, sizeof(int32_t) * (size_t)(S * V), hipMemcpyDeviceToHost, stream));
    CHECK_HIP(hipStreamSynchronize(stream));
    for (int64_t s = 0; s < S; ++s)
        for (int32_t v = 0; v < V; ++v)
            printf("state %lld v %d score %.9g next %d\n", (long long)s, v, h_scores[s * V + v], h_next[s * V + v]);

    /* greedy plain fusion at lambda = 0 along the sentence: the ASR row of step t
     * puts 0 on the sentence's token and -30 elsewhere, so the step takes it */
    float *h_asr = malloc(sizeof(float) * (size_t)V);
    float *d_asr;
    int32_t *d_tok, h_tok = -1, st = 0;
    CHECK_HIP(hipMalloc((void **)&d_asr, sizeof(float) * (size_t)V));
    CHECK_HIP(hipMalloc((void **)&d_tok, sizeof(int32_t)));
    CHECK_HIP(hipMemcpyAsync(d_states, &st, sizeof(int32_t), hipMemcpyHostToDevice, stream));
    int tok, t = 0;
    while (scanf("%d", &tok) == 1) {
        for (int32_t v = 0; v < V; ++v) h_asr[v] = v == tok ? 0.0f : -30.0f;
        CHECK_HIP(hipMemcpyAsync(d_asr, h_asr, sizeof(float) * (size_t)V, hipMemcpyHostToDevice, stream));
        CHECK_LM(ngpu_lm_fused_greedy_step(lm, d_asr, 1, V, NGPU_FUSION_PLAIN, 0.0f, d_states, NULL, d_tok, stream));
        CHECK_HIP(hipMemcpyAsync(&h_tok, d_tok, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
        CHECK_HIP(hipMemcpyAsync(&st, d_states, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
        CHECK_HIP(hipStreamSynchronize(stream));
        printf("step %d token %d state %d\n", t++, h_tok, st);
    }
    int64_t bad = -1;
    CHECK_LM(ngpu_lm_check_states(lm, stream, &bad));
    printf("bad states %lld\n", (long long)bad);

    /* an invalid call: a negative batch size is rejected before any launch */
    printf("error %d\n", ngpu_lm_advance(lm, d_states, -1, d_scores, d_next, stream));

    hipFree(d_asr);
    hipFree(d_tok);
    hipFree(d_states);
    hipFree(d_scores);
    hipFree(d_next);
    hipFree(img);
    hipStreamDestroy(stream);
    ngpu_lm_free(lm);
    free(order); free(tokens); free(W); free(B); free(h_states); free(h_scores); free(h_next); free(h_asr);
    printf("ok\n");
    return 0;
}
