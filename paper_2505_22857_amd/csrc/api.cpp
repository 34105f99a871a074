// C ABI entry points: argument checks, error reporting, upload and launches.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>

#include "trie.h"

namespace ngpu {
hipError_t launch_advance(const DevTrie &t, const int32_t *states, int64_t B, float *scores, int32_t *next,
                          hipStream_t stream);
hipError_t launch_fused_step(const DevTrie &t, const float *asr, int64_t B, int64_t ld, int mode, float lambda,
                             int32_t *states, int32_t *prev, int32_t *tokens, hipStream_t stream);
hipError_t launch_fused_decode(const DevTrie &t, const float *asr, int64_t B, int64_t T, int64_t sb, int64_t st,
                               const int32_t *lengths, int mode, float lambda, int32_t *states, int32_t *prev,
                               int32_t *labels, int32_t *label_states, hipStream_t stream);
hipError_t launch_final_weights(const DevTrie &t, const int32_t *states, int64_t B, float *out, hipStream_t stream);
hipError_t launch_fused_topk(const DevTrie &t, const float *asr, int64_t B, int64_t ld, float lambda, int k,
                             const int32_t *states, int32_t *tokens, float *scores, int32_t *next,
                             hipStream_t stream);
}  // namespace ngpu

namespace {

thread_local std::string g_last_error;

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

int ok() {
    g_last_error.clear();
    return NGPU_OK;
}

int hip_fail(hipError_t e, const char *what) {
    return fail(NGPU_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Largest batch whose grid fits the 32-bit dispatch size in work-items: 64
// per hypothesis (256 for the four-wavefront fused kernels, used up to 512
// hypotheses only).
constexpr int64_t kMaxBatch = NGPU_LM_MAX_BATCH;
static_assert(kMaxBatch * 64 <= int64_t(UINT32_MAX), "grid must fit the dispatch size");

ngpu::DevTrie dev_view(const ngpu_lm *lm) {
    const unsigned char *base = static_cast<const unsigned char *>(lm->dev);
    const ngpu::ImageHeader &h = lm->hdr;
    ngpu::DevTrie t;
    t.chain = base + h.off_chain;
    t.dense_w = reinterpret_cast<const float *>(base + h.off_dense_w);
    t.dense_to = reinterpret_cast<const int32_t *>(base + h.off_dense_to);
    t.arcs = reinterpret_cast<const ngpu::Arc *>(base + h.off_arcs);
    t.top_arcs = reinterpret_cast<const ngpu::TopArc *>(base + h.off_top_arcs);
    t.top_begin = int32_t(h.top_arc_begin);
    t.to_delta = h.arc_to_delta;
    t.final_w = h.has_final ? reinterpret_cast<const float *>(base + h.off_final) : nullptr;
    t.dense_c = h.off_dense_c ? reinterpret_cast<const float *>(base + h.off_dense_c) : nullptr;
    t.dense_base = h.off_dense_c ? reinterpret_cast<const int32_t *>(base + h.off_dense_base) : nullptr;
    t.compact_rank = h.compact_rank;
    t.status = reinterpret_cast<int32_t *>(const_cast<unsigned char *>(base) + h.off_status);
    t.num_states = int32_t(lm->S);
    t.vocab_size = lm->V;
    t.max_order = lm->N;
    for (int k = 0; k <= NGPU_LM_MAX_ORDER; ++k) t.first[k] = h.first[k];
    for (int k = 0; k < NGPU_LM_MAX_ORDER; ++k) t.off_order[k] = h.off_order[k];
    return t;
}

// A query needs the uploaded image on the current device: its kernels run on
// the current device and read the image through plain device pointers.
int ready(const ngpu_lm *lm) {
    if (!lm->dev) return fail(NGPU_E_NOT_UPLOADED, "trie not uploaded");
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return hip_fail(hipGetLastError(), "hipGetDevice");
    if (cur != lm->device)
        return fail(NGPU_E_INVALID_ARG, "the trie image lives on device %d but device %d is current", lm->device, cur);
    return NGPU_OK;
}

}  // namespace

int ngpu::set_error(int code, const std::string &msg) {
    g_last_error = msg;
    return code;
}

extern "C" {

const char *ngpu_lm_last_error(void) { return g_last_error.c_str(); }

int ngpu_lm_build(const ngpu_ngram_list *list, int32_t vocab_size, float unk_logprob, uint32_t flags,
                  ngpu_lm **out) {
    if (!out) return fail(NGPU_E_INVALID_ARG, "out is null");
    *out = nullptr;
    if (!list) return fail(NGPU_E_INVALID_ARG, "list is null");
    if ((flags & ~(NGPU_BUILD_BOS_EOS | NGPU_BUILD_REPAIR_CLOSURE)) != 0)
        return fail(NGPU_E_INVALID_ARG, "unknown build flags");
    ngpu_lm *lm = new (std::nothrow) ngpu_lm();
    if (!lm) return fail(NGPU_E_NO_MEMORY, "handle allocation failed");
    std::string err;
    int rc;
    try {
        rc = ngpu::build_trie(list, vocab_size, unk_logprob, flags, lm, &err);
    } catch (const std::bad_alloc &) {
        rc = NGPU_E_NO_MEMORY;
        err = "host allocation failed while building the trie";
    }
    if (rc != NGPU_OK) {
        delete lm;
        return fail(rc, "%s", err.c_str());
    }
    *out = lm;
    return ok();
}

void ngpu_lm_free(ngpu_lm *lm) { delete lm; }

int ngpu_lm_info(const ngpu_lm *lm, ngpu_lm_info_t *out) {
    if (!lm || !out) return fail(NGPU_E_INVALID_ARG, "null argument");
    out->num_states = lm->S;
    out->num_arcs = lm->A;
    out->max_order = lm->N;
    out->vocab_size = lm->V;
    out->device_bytes = int64_t(lm->image.size());
    return ok();
}

int ngpu_lm_state_context(const ngpu_lm *lm, int64_t state, int32_t *tokens_out, int32_t *order_out) {
    if (!lm || !order_out || (!tokens_out && lm->N > 1)) return fail(NGPU_E_INVALID_ARG, "null argument");
    if (state < 0 || state >= lm->S) return fail(NGPU_E_BAD_STATE, "state %lld outside [0, %lld)",
                                                 (long long)state, (long long)lm->S);
    int32_t k = 0;
    for (int64_t s = state; s != 0; s = lm->state_parent[size_t(s)]) ++k;
    *order_out = k;
    int64_t s = state;
    for (int32_t i = k - 1; i >= 0; --i) {
        tokens_out[i] = lm->state_tok[size_t(s)];
        s = lm->state_parent[size_t(s)];
    }
    return ok();
}

size_t ngpu_lm_device_bytes(const ngpu_lm *lm) { return lm ? lm->image.size() : 0; }

int ngpu_lm_start_state(const ngpu_lm *lm, int64_t *state) {
    if (!lm || !state) return fail(NGPU_E_INVALID_ARG, "null argument");
    *state = lm->hdr.start_state;
    return ok();
}

int ngpu_lm_final_weights(const ngpu_lm *lm, const int32_t *d_states, int64_t B, float *d_final,
                          void *hip_stream) {
    if (!lm) return fail(NGPU_E_INVALID_ARG, "null handle");
    if (!lm->hdr.has_final) return fail(NGPU_E_INVALID_ARG, "the model has no </s> (build with NGPU_BUILD_BOS_EOS)");
    if (const int rc = ready(lm)) return rc;
    if (B < 0 || B > kMaxBatch) return fail(NGPU_E_INVALID_ARG, "B = %lld out of range", (long long)B);
    if (B == 0) return ok();
    if (!d_states || !d_final) return fail(NGPU_E_INVALID_ARG, "null device pointer");
    hipError_t e = ngpu::launch_final_weights(dev_view(lm), d_states, B, d_final,
                                              static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return hip_fail(e, "final weights launch");
    return ok();
}

int ngpu_lm_upload(ngpu_lm *lm, void *dev_buf, size_t dev_bytes, void *hip_stream) {
    if (!lm || !dev_buf) return fail(NGPU_E_INVALID_ARG, "null argument");
    if (reinterpret_cast<uintptr_t>(dev_buf) % ngpu::kAlign != 0)
        return fail(NGPU_E_INVALID_ARG, "device buffer must be 256-byte aligned");
    if (dev_bytes < lm->image.size())
        return fail(NGPU_E_INVALID_ARG, "device buffer has %zu bytes, the image needs %zu", dev_bytes,
                    lm->image.size());
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, dev_buf);
    if (e != hipSuccess || attr.type != hipMemoryTypeDevice) {
        (void)hipGetLastError();
        return fail(NGPU_E_INVALID_ARG, "dev_buf is not device memory");
    }
    e = hipMemcpyAsync(dev_buf, lm->image.data(), lm->image.size(), hipMemcpyHostToDevice,
                       static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (upload)");
    lm->dev = dev_buf;
    lm->device = attr.device;
    return ok();
}

int ngpu_lm_advance(const ngpu_lm *lm, const int32_t *d_states, int64_t B, float *d_scores, int32_t *d_next,
                    void *hip_stream) {
    if (!lm) return fail(NGPU_E_INVALID_ARG, "null handle");
    if (const int rc = ready(lm)) return rc;
    if (B < 0 || B > kMaxBatch) return fail(NGPU_E_INVALID_ARG, "B = %lld outside [0, %lld]", (long long)B,
                                            (long long)kMaxBatch);
    if (B == 0) return ok();
    if (!d_states || !d_scores || !d_next) return fail(NGPU_E_INVALID_ARG, "null device pointer");
    const ngpu::DevTrie t = dev_view(lm);
    hipError_t e = ngpu::launch_advance(t, d_states, B, d_scores, d_next, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return hip_fail(e, "advance launch");
    return ok();
}

int ngpu_lm_fused_greedy_step(const ngpu_lm *lm, const float *d_asr, int64_t B, int64_t asr_ld, int32_t mode,
                              float lambda, int32_t *d_states, int32_t *d_prev, int32_t *d_tokens,
                              void *hip_stream) {
    if (!lm) return fail(NGPU_E_INVALID_ARG, "null handle");
    if (const int rc = ready(lm)) return rc;
    if (mode < NGPU_FUSION_PLAIN || mode > NGPU_FUSION_AED)
        return fail(NGPU_E_INVALID_ARG, "unknown fusion mode %d", mode);
    if (mode == NGPU_FUSION_AED && !lm->hdr.has_final)
        return fail(NGPU_E_INVALID_ARG, "AED fusion needs a model with </s> (NGPU_BUILD_BOS_EOS)");
    if (B < 0 || B > kMaxBatch) return fail(NGPU_E_INVALID_ARG, "B = %lld outside [0, %lld]", (long long)B,
                                            (long long)kMaxBatch);
    const int64_t need = mode == NGPU_FUSION_PLAIN ? lm->V : int64_t(lm->V) + 1;
    if (asr_ld < need) return fail(NGPU_E_INVALID_ARG, "asr_ld %lld < %lld", (long long)asr_ld, (long long)need);
    if (!std::isfinite(lambda)) return fail(NGPU_E_INVALID_ARG, "lambda must be finite");
    if (B == 0) return ok();
    if (!d_asr || !d_states || !d_tokens || (mode == NGPU_FUSION_CTC && !d_prev))
        return fail(NGPU_E_INVALID_ARG, "null device pointer");
    const ngpu::DevTrie t = dev_view(lm);
    hipError_t e = ngpu::launch_fused_step(t, d_asr, B, asr_ld, mode, lambda, d_states, d_prev, d_tokens,
                                           static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return hip_fail(e, "fused step launch");
    return ok();
}

int ngpu_lm_fused_topk(const ngpu_lm *lm, const float *d_asr, int64_t B, int64_t asr_ld, float lambda, int32_t k,
                       const int32_t *d_states, int32_t *d_tokens, float *d_scores, int32_t *d_next,
                       void *hip_stream) {
    if (!lm) return fail(NGPU_E_INVALID_ARG, "null handle");
    if (const int rc = ready(lm)) return rc;
    if (B < 0 || B > kMaxBatch) return fail(NGPU_E_INVALID_ARG, "B = %lld outside [0, %lld]", (long long)B,
                                            (long long)kMaxBatch);
    if (k < 1 || k > lm->V || k > NGPU_LM_MAX_TOPK)
        return fail(NGPU_E_INVALID_ARG, "k = %d outside [1, min(V, %d)]", k, NGPU_LM_MAX_TOPK);
    if (asr_ld < lm->V) return fail(NGPU_E_INVALID_ARG, "asr_ld %lld < V", (long long)asr_ld);
    if (!std::isfinite(lambda)) return fail(NGPU_E_INVALID_ARG, "lambda must be finite");
    if (B == 0) return ok();
    if (!d_asr || !d_states || !d_tokens || !d_scores || !d_next)
        return fail(NGPU_E_INVALID_ARG, "null device pointer");
    const ngpu::DevTrie t = dev_view(lm);
    hipError_t e = ngpu::launch_fused_topk(t, d_asr, B, asr_ld, lambda, k, d_states, d_tokens, d_scores, d_next,
                                           static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return hip_fail(e, "fused top-k launch");
    return ok();
}

int ngpu_lm_fused_greedy_decode(const ngpu_lm *lm, const float *d_asr, int64_t B, int64_t T, int64_t stride_b,
                                int64_t stride_t, const int32_t *d_lengths, int32_t mode, float lambda,
                                int32_t *d_states, int32_t *d_prev, int32_t *d_labels, int32_t *d_label_states,
                                void *hip_stream) {
    if (!lm) return fail(NGPU_E_INVALID_ARG, "null handle");
    if (const int rc = ready(lm)) return rc;
    if (mode < NGPU_FUSION_PLAIN || mode > NGPU_FUSION_AED)
        return fail(NGPU_E_INVALID_ARG, "unknown fusion mode %d", mode);
    if (mode == NGPU_FUSION_AED && !lm->hdr.has_final)
        return fail(NGPU_E_INVALID_ARG, "AED fusion needs a model with </s> (NGPU_BUILD_BOS_EOS)");
    if (B < 0 || B > kMaxBatch || T < 0)
        return fail(NGPU_E_INVALID_ARG, "bad sizes B=%lld (at most %lld) T=%lld", (long long)B, (long long)kMaxBatch,
                    (long long)T);
    if (stride_b < 0 || stride_t < 0) return fail(NGPU_E_INVALID_ARG, "negative strides");
    const int64_t need = mode == NGPU_FUSION_PLAIN ? lm->V : int64_t(lm->V) + 1;
    if (T > 1 && stride_t < need) return fail(NGPU_E_INVALID_ARG, "stride_t %lld < %lld", (long long)stride_t,
                                              (long long)need);
    if (B > 1 && stride_b < need) return fail(NGPU_E_INVALID_ARG, "stride_b %lld < %lld", (long long)stride_b,
                                              (long long)need);
    if (!std::isfinite(lambda)) return fail(NGPU_E_INVALID_ARG, "lambda must be finite");
    if (B == 0 || T == 0) return ok();
    if (!d_asr || !d_states || !d_labels || (mode == NGPU_FUSION_CTC && !d_prev))
        return fail(NGPU_E_INVALID_ARG, "null device pointer");
    const ngpu::DevTrie t = dev_view(lm);
    hipError_t e = ngpu::launch_fused_decode(t, d_asr, B, T, stride_b, stride_t, d_lengths, mode, lambda, d_states,
                                             d_prev, d_labels, d_label_states, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return hip_fail(e, "fused decode launch");
    return ok();
}

int ngpu_lm_check_states(const ngpu_lm *lm, void *hip_stream, int64_t *bad_count) {
    if (!lm) return fail(NGPU_E_INVALID_ARG, "null handle");
    if (const int rc = ready(lm)) return rc;
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    int32_t host[4] = {0, 0, 0, 0};
    void *dstatus = static_cast<unsigned char *>(lm->dev) + lm->hdr.off_status;
    hipError_t e = hipMemcpyAsync(host, dstatus, sizeof host, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "reading the status word");
    if (host[0] != 0) {
        const int32_t zero[4] = {0, 0, 0, 0};
        e = hipMemcpyAsync(dstatus, zero, sizeof zero, hipMemcpyHostToDevice, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        if (e != hipSuccess) return hip_fail(e, "clearing the status word");
    }
    if (bad_count) *bad_count = host[0];
    if (host[0] != 0) return fail(NGPU_E_BAD_STATE, "%d out-of-range input states", host[0]);
    return ok();
}

int ngpu_lm_sync_check(const ngpu_lm *lm, void *hip_stream) {
    int64_t bad = 0;
    return ngpu_lm_check_states(lm, hip_stream, &bad);
}

int ngpu_lm_host_image(const ngpu_lm *lm, const void **data, size_t *bytes) {
    if (!lm || !data || !bytes) return fail(NGPU_E_INVALID_ARG, "null argument");
    *data = lm->image.data();
    *bytes = lm->image.size();
    return ok();
}

int ngpu_lm_query_bytes(const ngpu_lm *lm, const int32_t *h_states, int64_t B, int64_t *hbm_bytes,
                        int64_t *total_bytes) {
    if (!lm || (B > 0 && !h_states) || !hbm_bytes || !total_bytes) return fail(NGPU_E_INVALID_ARG, "null argument");
    const int64_t V = lm->V;
    int64_t hbm = 0, total = 0;
    for (int64_t b = 0; b < B; ++b) {
        int64_t s = h_states[b];
        if (s < 0 || s >= lm->S) return fail(NGPU_E_BAD_STATE, "state %lld out of range", (long long)s);
        int k = 0;   // order of s
        for (int j = 1; j < lm->N; ++j)
            if (s >= lm->hdr.first[j]) k = j;
        int64_t bytes = 8 * V + 16 * (k > 0 ? k : 1);   // output row + chain record
        for (int j = 0; j < k - 1; ++j) {                // sparse levels: orders k..2
            bytes += 12 * int64_t(lm->rec[size_t(s)].end - lm->rec[size_t(s)].begin);
            s = lm->rec[size_t(s)].bto;
        }
        hbm += bytes;
        total += bytes + 8 * V;                          // + the shared dense row
    }
    *hbm_bytes = hbm;
    *total_bytes = total;
    return ok();
}

}  // extern "C"
