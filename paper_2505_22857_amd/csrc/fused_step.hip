// Greedy shallow fusion (Section 2.3): one step over a batch of hypotheses, and
// a whole decode over all frames of a batch of utterances in one launch.
//
// One wavefront per hypothesis.  CTC and transducer modes first take the plain
// ASR argmax over the V + 1 classes; when that keeps blank (or, for CTC, the
// previous label) the LM is not consulted at all and the state stays.
// Otherwise the wavefront walks its state's backoff chain into an LDS row (the
// same walk as the advance kernel, with no HBM write of the row), merges the
// dense row of the order-1 ancestor, forms fmaf(lambda, lm[v], asr[v]) per
// token and takes the argmax with lowest-index ties: each lane keeps a running
// maximum over its tokens (read four at a time from LDS), then one 64-bit key
// (value, ~index) per lane is reduced across the wavefront with DPP moves.
// The winner's next state comes from the same merge.  No MFMA: one fma and one
// compare per token.
//
// The decode kernel keeps each utterance's state and previous label in
// registers across frames: frame t + 1 depends on frame t only through them,
// so a single launch replaces T launches and their host round trips.
//
// AED mode (Section 2.3): class V is <eos>, whose LM score is the state's
// final weight (the </s> score, precomputed per state); <eos> keeps the state.
#include <hip/hip_runtime.h>

#include "walk.h"

namespace ngpu {

enum { kPlain = 0, kCtc = 1, kTransducer = 2, kAed = 3 };

// Words of an ASR row buffer in LDS: the V + 1 classes rounded up to whole
// 256-word stripes, so that the 16-byte reads of the scans stay inside it.
__host__ __device__ inline int asr_row_words(int V) { return lds_row(V + 1); }

// Per-lane argmax of row[v] over tokens v < V.  Tokens go in stripes of 256:
// lane l reads 4 consecutive tokens 4l .. 4l + 3 of each stripe with one
// 16-byte LDS read, so every lane meets its tokens in ascending order.
__device__ __forceinline__ void scan_row(const float *row, int V, int lane, float &bx, int &bi) {
    const int full = V & ~255;
#pragma unroll 4
    for (int c = 0; c < full; c += 256) {
        const int v0 = c + 4 * lane;
        const f32x4 a = *reinterpret_cast<const f32x4 *>(row + v0);
#pragma unroll
        for (int j = 0; j < 4; ++j) take_max(a[j], v0 + j, bx, bi);
    }
    if (full < V) {
        const int v0 = full + 4 * lane;
        const f32x4 a = *reinterpret_cast<const f32x4 *>(row + v0);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (v0 + j < V) take_max(a[j], v0 + j, bx, bi);
    }
}

// Per-lane argmax of fmaf(lambda, lm[v], row[v]) over tokens v < V (v != pv
// in CTC mode), lm[v] from the walked LDS row; same stripes as scan_row.
template <int MODE>
__device__ __forceinline__ void scan_fused(const ChainHead &h, const float *ls, const int *ln, const float *row,
                                           float lambda, int pv, int V, int lane, float &bx, int &bi) {
    auto four = [&](int v0, bool tail) {
        const f32x4 x = *reinterpret_cast<const f32x4 *>(ls + v0);
        const i32x4 n = *reinterpret_cast<const i32x4 *>(ln + v0);
        const f32x4 a = *reinterpret_cast<const f32x4 *>(row + v0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float lm;
            int nx;
            slot_value(h, x[j], n[j], lm, nx);
            const float f = __builtin_fmaf(lambda, lm, a[j]);
            const int v = v0 + j;
            if ((MODE != kCtc || v != pv) && (!tail || v < V)) take_max(f, v, bx, bi);
        }
    };
    const int full = V & ~255;
#pragma unroll 4
    for (int c = 0; c < full; c += 256) four(c + 4 * lane, false);
    if (full < V) four(full + 4 * lane, true);
}

// One fused greedy step of the wavefront's hypothesis.  row: its V + 1 ASR
// log-probabilities in LDS (asr_row_words(V) words); they have landed unless
// ROW_PENDING, in which case their copy was issued just before.  s: valid
// state (uniform); pv: previous label (CTC).  Returns the label and updates s.
// All lanes return the same values.
template <int MODE, bool ROW_PENDING>
__device__ __forceinline__ int greedy_step(const DevTrie &t, const float *row, float lambda, int &s, int pv,
                                           float *ls, int *ln, int lane, const float *pf_src = nullptr,
                                           float *pf_dst = nullptr, int pf_n = 0) {
    const int V = t.vocab_size;
    const float fin = MODE == kAed ? t.final_w[s] : 0.0f;   // <eos> takes the state's final weight
    // The chain record is fetched first: in CTC and transducer modes its load
    // overlaps the plain ASR argmax, which may still find that the LM is not needed.
    int nlev;
    const int4 rec = fetch_record(t, s, lane, nlev);
    if (MODE == kCtc || MODE == kTransducer) {
        if (ROW_PENDING) wait_lds_copies();
        float bx = -__builtin_inff(), av;
        int bi = kNone;
        scan_row(row, V, lane, bx, bi);
        int a = wave_argmax(bx, bi, av);
        if (a == kNone) a = 0;                    // every token at -inf: the first one, unless blank beats it
        if (row[V] > av) a = V;                   // blank only when strictly larger (it has the highest index)
        if (a == V || (MODE == kCtc && a == pv)) {   // blank or repeat: no LM, no move
            if (pf_src) copy_to_lds_dword(pf_src, pf_dst, pf_n, lane);
            return a;
        }
    }
    const ChainHead h = walk_record(t, rec, nlev, ls, ln, lane, pf_src, pf_dst, pf_n);
    float bx = -__builtin_inff(), wv;
    int bi = kNone;
    scan_fused<MODE>(h, ls, ln, row, lambda, pv, V, lane, bx, bi);
    int w = wave_argmax(bx, bi, wv);
    if (w == kNone) w = (MODE == kCtc && pv == 0) ? 1 : 0;   // every candidate at -inf: the first one
    if (MODE == kAed && __builtin_fmaf(lambda, fin, row[V]) > wv)
        return V;   // <eos> strictly above every token: the sentence ends, the state stays
    float lm;
    int n;
    slot_value(h, ls[w], ln[w], lm, n);   // uniform w: every lane reads the same slot
    s = n;
    return w;
}

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
    float *ls = lds + size_t(wave) * (2 * lds_row(V) + asr_row_words(V));
    int *ln = reinterpret_cast<int *>(ls + lds_row(V));
    float *arow = reinterpret_cast<float *>(ln + lds_row(V));

    // the ASR row's copy into LDS goes out with the state load
    copy_to_lds_dword(asr + b * ld, arow, MODE == kPlain ? V : V + 1, lane);
    int s = __builtin_amdgcn_readfirstlane(states[b]);
    if (s < 0 || s >= t.num_states) {
        if (lane == 0) {
            atomicAdd(&t.status[0], 1);
            tokens[b] = -1;
        }
        wait_lds_copies();   // no copy into LDS outlives the wavefront
        return;
    }
    const int pv = MODE == kCtc ? __builtin_amdgcn_readfirstlane(prev[b]) : -1;
    const int label = greedy_step<MODE, true>(t, arow, lambda, s, pv, ls, ln, lane);
    if (lane == 0) {
        tokens[b] = label;
        states[b] = s;
        if (MODE == kCtc) prev[b] = label;
    }
}

// Whole greedy decode: utterance b runs frames 0 .. len_b - 1 of
// asr[b * stride_b + t * stride_t + class].
template <int MODE>
__global__ __launch_bounds__(kWave) void fused_decode_kernel(DevTrie t, const float *__restrict__ asr, int64_t B,
                                                              int64_t T, int64_t stride_b, int64_t stride_t,
                                                              const int32_t *__restrict__ lengths, float lambda,
                                                              int32_t *__restrict__ states,
                                                              int32_t *__restrict__ prev,
                                                              int32_t *__restrict__ labels,
                                                              int32_t *__restrict__ label_states) {
    extern __shared__ float lds[];
    const int lane = threadIdx.x;
    const int64_t b = blockIdx.x;
    if (b >= B) return;
    const int V = t.vocab_size;
    const int rowp = asr_row_words(V);
    float *ls = lds;
    int *ln = reinterpret_cast<int *>(ls + lds_row(V));
    float *abuf = reinterpret_cast<float *>(ln + lds_row(V));   // two ASR rows, double-buffered
    int32_t *lab = labels + b * T;
    int32_t *lst = label_states ? label_states + b * T : nullptr;

    int64_t len = T;
    if (lengths) {
        len = __builtin_amdgcn_readfirstlane(lengths[b]);
        len = len < 0 ? 0 : (len > T ? T : len);
    }
    int s = __builtin_amdgcn_readfirstlane(states[b]);
    if (s < 0 || s >= t.num_states) {
        if (lane == 0) atomicAdd(&t.status[0], 1);
        for (int64_t f = lane; f < T; f += kWave) {
            lab[f] = -1;
            if (lst) lst[f] = -1;
        }
        return;
    }
    int pv = MODE == kCtc ? __builtin_amdgcn_readfirstlane(prev[b]) : -1;
    const float *row = asr + b * stride_b;
    const int cn = MODE == kPlain ? V : V + 1;   // ASR row words used
    if (len > 0) copy_to_lds_dword(row, abuf, cn, lane);
    for (int64_t f = 0; f < len; ++f, row += stride_t) {
        // frame f reads its ASR row from LDS, copied during frame f - 1 (or
        // before the loop); the walk also starts the copy of row f + 1
        wait_lds_copies();
        float *cur = abuf + (f & 1) * rowp;
        float *nxt = abuf + ((f + 1) & 1) * rowp;
        const float *pf = f + 1 < len ? row + stride_t : nullptr;
        const int label = greedy_step<MODE, false>(t, cur, lambda, s, pv, ls, ln, lane, pf, nxt, cn);
        if (MODE == kCtc) pv = label;
        if (lane == 0) {
            lab[f] = label;
            if (lst) lst[f] = s;
        }
    }
    for (int64_t f = len + lane; f < T; f += kWave) {   // frames past the utterance's end
        lab[f] = -1;
        if (lst) lst[f] = s;
    }
    if (lane == 0) {
        states[b] = s;
        if (MODE == kCtc) prev[b] = pv;
    }
}

// The k best fused scores of one hypothesis per wavefront (beam-search
// expansion): the row of fused values fmaf(lambda, lm[v], asr[v]) stays in
// LDS, and k rounds of the wave argmax each take the best token not yet taken
// (bit 31 of its next-state slot marks it).  Cost O(k V / 64) per wavefront.
__global__ __launch_bounds__(kWave) void fused_topk_kernel(DevTrie t, const float *__restrict__ asr, int64_t B,
                                                           int64_t ld, float lambda, int k,
                                                           const int32_t *__restrict__ states,
                                                           int32_t *__restrict__ tokens, float *__restrict__ scores,
                                                           int32_t *__restrict__ next) {
    extern __shared__ float lds[];
    const int lane = threadIdx.x;
    const int64_t b = blockIdx.x;
    if (b >= B) return;
    const int V = t.vocab_size;
    float *ls = lds;
    int *ln = reinterpret_cast<int *>(ls + lds_row(V));
    int32_t *otok = tokens + b * k;
    float *osc = scores + b * k;
    int32_t *onx = next + b * k;
    const int s = __builtin_amdgcn_readfirstlane(states[b]);
    if (s < 0 || s >= t.num_states) {
        if (lane == 0) atomicAdd(&t.status[0], 1);
        for (int j = lane; j < k; j += kWave) {
            otok[j] = -1;
            osc[j] = NAN;
            onx[j] = -1;
        }
        return;
    }
    const ChainHead h = walk_into_lds(t, s, ls, ln, lane);
    const float *row = asr + b * ld;
    for (int v = lane; v < V; v += kWave) {   // each lane rewrites only its own slots
        float lm;
        int n;
        slot_value(h, ls[v], ln[v], lm, n);
        ls[v] = __builtin_fmaf(lambda, lm, row[v]);
        ln[v] = n;
    }
    for (int j = 0; j < k; ++j) {
        unsigned long long best = 0;
        for (int v = lane; v < V; v += kWave) {
            if (ln[v] >= 0) {
                const unsigned long long key = argmax_key(ls[v], v);
                best = key > best ? key : best;
            }
        }
        const int w = argmax_index(wave_max_u64(best));
        if (lane == 0) {
            otok[j] = w;
            osc[j] = ls[w];
            onx[j] = ln[w];
            ln[w] = ln[w] | int32_t(0x80000000u);
        }
    }
}

__global__ __launch_bounds__(256) void final_weights_kernel(DevTrie t, const int32_t *__restrict__ states, int64_t B,
                                                          float *__restrict__ out) {
    const int64_t b = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (b >= B) return;
    const int s = states[b];
    if (s < 0 || s >= t.num_states) {
        atomicAdd(&t.status[0], 1);
        out[b] = NAN;
        return;
    }
    out[b] = t.final_w[s];
}

hipError_t launch_final_weights(const DevTrie &t, const int32_t *states, int64_t B, float *out, hipStream_t stream) {
    hipLaunchKernelGGL(final_weights_kernel, dim3(unsigned((B + 255) / 256)), dim3(256), 0, stream, t, states, B,
                       out);
    return hipGetLastError();
}

hipError_t launch_fused_topk(const DevTrie &t, const float *asr, int64_t B, int64_t ld, float lambda, int k,
                             const int32_t *states, int32_t *tokens, float *scores, int32_t *next,
                             hipStream_t stream) {
    const size_t lds = 2 * size_t(lds_row(t.vocab_size)) * sizeof(float);
    hipLaunchKernelGGL(fused_topk_kernel, dim3(unsigned(B)), dim3(kWave), lds, stream, t, asr, B, ld, lambda, k,
                       states, tokens, scores, next);
    return hipGetLastError();
}

template <int HPB, int MODE>
static hipError_t launch_one(const DevTrie &t, const float *asr, int64_t B, int64_t ld, float lambda,
                             int32_t *states, int32_t *prev, int32_t *tokens, hipStream_t stream) {
    const int64_t blocks = (B + HPB - 1) / HPB;
    const size_t lds =
        size_t(HPB) * (2 * size_t(lds_row(t.vocab_size)) + size_t(asr_row_words(t.vocab_size))) * sizeof(float);
    hipLaunchKernelGGL((fused_step_kernel<HPB, MODE>), dim3(unsigned(blocks)), dim3(HPB * kWave), lds, stream,
                       t, asr, B, ld, lambda, states, prev, tokens);
    return hipGetLastError();
}

// One hypothesis per workgroup: a step batch is a few hundred hypotheses, so
// spreading them over all CUs beats packing them.
hipError_t launch_fused_step(const DevTrie &t, const float *asr, int64_t B, int64_t ld, int mode, float lambda,
                             int32_t *states, int32_t *prev, int32_t *tokens, hipStream_t stream) {
    switch (mode) {
        case kPlain: return launch_one<1, kPlain>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        case kCtc: return launch_one<1, kCtc>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        case kAed: return launch_one<1, kAed>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        default: return launch_one<1, kTransducer>(t, asr, B, ld, lambda, states, prev, tokens, stream);
    }
}

template <int MODE>
static hipError_t launch_decode_mode(const DevTrie &t, const float *asr, int64_t B, int64_t T, int64_t sb,
                                     int64_t st, const int32_t *lengths, float lambda, int32_t *states,
                                     int32_t *prev, int32_t *labels, int32_t *label_states, hipStream_t stream) {
    const size_t lds = (2 * size_t(lds_row(t.vocab_size)) + 2 * size_t(asr_row_words(t.vocab_size))) * sizeof(float);
    hipLaunchKernelGGL((fused_decode_kernel<MODE>), dim3(unsigned(B)), dim3(kWave), lds, stream, t, asr, B, T, sb,
                       st, lengths, lambda, states, prev, labels, label_states);
    return hipGetLastError();
}

hipError_t launch_fused_decode(const DevTrie &t, const float *asr, int64_t B, int64_t T, int64_t sb, int64_t st,
                               const int32_t *lengths, int mode, float lambda, int32_t *states, int32_t *prev,
                               int32_t *labels, int32_t *label_states, hipStream_t stream) {
    switch (mode) {
        case kPlain:
            return launch_decode_mode<kPlain>(t, asr, B, T, sb, st, lengths, lambda, states, prev, labels,
                                              label_states, stream);
        case kCtc:
            return launch_decode_mode<kCtc>(t, asr, B, T, sb, st, lengths, lambda, states, prev, labels,
                                            label_states, stream);
        case kAed:
            return launch_decode_mode<kAed>(t, asr, B, T, sb, st, lengths, lambda, states, prev, labels,
                                            label_states, stream);
        default:
            return launch_decode_mode<kTransducer>(t, asr, B, T, sb, st, lengths, lambda, states, prev, labels,
                                                   label_states, stream);
    }
}

}  // namespace ngpu
