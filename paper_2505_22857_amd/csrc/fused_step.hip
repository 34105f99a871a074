// One greedy shallow-fusion step (Section 2.3) over a batch of hypotheses.
//
// One wavefront per hypothesis.  CTC and transducer modes first take the plain
// ASR argmax over the V + 1 classes; when that keeps blank (or, for CTC, the
// previous label) the LM is not consulted at all and the state stays.
// Otherwise the wavefront walks its state's backoff chain into an LDS row (the
// same walk as the advance kernel, with no HBM write of the row), merges the
// dense row of the order-1 ancestor, forms fmaf(lambda, lm[v], asr[v]) per
// token and reduces to the argmax with lowest-index ties through 64-bit keys
// (value, ~index) and cross-lane shuffles.  The winner's next state comes from
// the same merge.  No MFMA: one fma and one compare per token.
#include <hip/hip_runtime.h>

#include "walk.h"

namespace ngpu {

enum { kPlain = 0, kCtc = 1, kTransducer = 2 };

template <int HPB, int MODE>
__global__ __launch_bounds__(HPB * kWave) void fused_step_kernel(DevTrie t, const float *__restrict__ asr,
                                                                  int64_t B, int64_t ld, float lambda,
                                                                  int32_t *__restrict__ states,
                                                                  int32_t *__restrict__ prev,
                                                                  int32_t *__restrict__ tokens) {
    extern __shared__ float lds[];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int64_t b = int64_t(blockIdx.x) * HPB + wave;
    if (b >= B) return;
    const int V = t.vocab_size;
    float *ls = lds + size_t(wave) * 2 * V;
    int *ln = reinterpret_cast<int *>(ls + V);
    const float *row = asr + b * ld;

    const int s = __builtin_amdgcn_readfirstlane(states[b]);
    if (s < 0 || s >= t.num_states) {
        if (lane == 0) {
            atomicAdd(&t.status[0], 1);
            tokens[b] = -1;
        }
        return;
    }
    int pv = -1;
    if (MODE == kCtc) pv = __builtin_amdgcn_readfirstlane(prev[b]);

    if (MODE != kPlain) {
        unsigned long long best = 0;
        for (int v = lane; v <= V; v += kWave) {
            const unsigned long long k = argmax_key(row[v], v);
            best = k > best ? k : best;
        }
        const int a = argmax_index(wave_max_u64(best));
        if (a == V || (MODE == kCtc && a == pv)) {
            if (lane == 0) {
                tokens[b] = a;
                if (MODE == kCtc) prev[b] = a;
            }
            return;
        }
    }

    const ChainHead h = walk_into_lds(t, s, ls, ln, lane);
    const float *dw = t.dense_w + size_t(h.dense_row) * V;
    const int32_t *dt = t.dense_to + size_t(h.dense_row) * V;
    unsigned long long best = 0;
    for (int v = lane; v < V; v += kWave) {
        float lm;
        int n;
        merge_slot(h, ls[v], ln[v], dw[v], dt[v], lm, n);
        const float f = __builtin_fmaf(lambda, lm, row[v]);
        if (MODE == kCtc && v == pv) continue;
        const unsigned long long k = argmax_key(f, v);
        best = k > best ? k : best;
    }
    const int w = argmax_index(wave_max_u64(best));
    if (lane == 0) {
        float lm;
        int n;
        merge_slot(h, ls[w], ln[w], dw[w], dt[w], lm, n);
        states[b] = n;
        tokens[b] = w;
        if (MODE == kCtc) prev[b] = w;
    }
}

template <int HPB, int MODE>
static hipError_t launch_one(const DevTrie &t, const float *asr, int64_t B, int64_t ld, float lambda,
                             int32_t *states, int32_t *prev, int32_t *tokens, hipStream_t stream) {
    const int64_t blocks = (B + HPB - 1) / HPB;
    const size_t lds = size_t(HPB) * 2 * size_t(t.vocab_size) * sizeof(float);
    hipLaunchKernelGGL((fused_step_kernel<HPB, MODE>), dim3(unsigned(blocks)), dim3(HPB * kWave), lds, stream,
                       t, asr, B, ld, lambda, states, prev, tokens);
    return hipGetLastError();
}

int advance_rows_per_block(int V);

template <int MODE>
static hipError_t launch_mode(const DevTrie &t, const float *asr, int64_t B, int64_t ld, float lambda,
                              int32_t *states, int32_t *prev, int32_t *tokens, hipStream_t stream) {
    switch (advance_rows_per_block(t.vocab_size)) {
        case 4: return launch_one<4, MODE>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        case 2: return launch_one<2, MODE>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        default: return launch_one<1, MODE>(t, asr, B, ld, lambda, states, prev, tokens, stream);
    }
}

hipError_t launch_fused_step(const DevTrie &t, const float *asr, int64_t B, int64_t ld, int mode, float lambda,
                             int32_t *states, int32_t *prev, int32_t *tokens, hipStream_t stream) {
    switch (mode) {
        case kPlain: return launch_mode<kPlain>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        case kCtc: return launch_mode<kCtc>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        default: return launch_mode<kTransducer>(t, asr, B, ld, lambda, states, prev, tokens, stream);
    }
}

}  // namespace ngpu
