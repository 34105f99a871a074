// Batched full-vocabulary backoff query (Algorithm 1, batched over hypotheses).
//
// Grid: one wavefront per hypothesis, HPB wavefronts per workgroup, each with
// its own V-wide score/state row in LDS (8 bytes per token).  After the
// sparse levels are scattered, the row is merged with the order-1 ancestor's
// dense row and written to HBM with 16-byte stores (when V is a multiple of
// 4): lane l covers tokens 4l..4l+3 of each 256-token stripe, so one store
// instruction of the wavefront writes 1 KiB contiguously.  No MFMA: the work
// is gathers, scatters and one fp32 add per token.
#include <hip/hip_runtime.h>

#include <cmath>

#include "walk.h"

namespace ngpu {

template <int HPB, bool VEC>
__global__ __launch_bounds__(HPB * kWave) void advance_kernel(DevTrie t, const int32_t *__restrict__ states,
                                                               int64_t B, float *__restrict__ scores,
                                                               int32_t *__restrict__ next) {
    extern __shared__ float lds[];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int64_t b = int64_t(blockIdx.x) * HPB + wave;
    if (b >= B) return;  // whole wavefronts leave; no workgroup barrier is used
    const int V = t.vocab_size;
    float *ls = lds + size_t(wave) * 2 * V;
    int *ln = reinterpret_cast<int *>(ls + V);
    float *orow = scores + b * V;
    int32_t *nrow = next + b * V;

    const int s = __builtin_amdgcn_readfirstlane(states[b]);
    if (s < 0 || s >= t.num_states) {
        if (lane == 0) atomicAdd(&t.status[0], 1);
        for (int v = lane; v < V; v += kWave) {
            orow[v] = NAN;
            nrow[v] = -1;
        }
        return;
    }
    const ChainHead h = walk_into_lds(t, s, ls, ln, lane);
    const float *dw = t.dense_w + size_t(h.dense_row) * V;
    const int32_t *dt = t.dense_to + size_t(h.dense_row) * V;

    if (VEC) {
        for (int v = lane * 4; v < V; v += 4 * kWave) {
            const int4 n4 = *reinterpret_cast<const int4 *>(ln + v);
            const float4 x4 = *reinterpret_cast<const float4 *>(ls + v);
            const float4 w4 = *reinterpret_cast<const float4 *>(dw + v);
            const int4 t4 = *reinterpret_cast<const int4 *>(dt + v);
            float4 xo;
            int4 no;
            merge_slot(h, x4.x, n4.x, w4.x, t4.x, xo.x, no.x);
            merge_slot(h, x4.y, n4.y, w4.y, t4.y, xo.y, no.y);
            merge_slot(h, x4.z, n4.z, w4.z, t4.z, xo.z, no.z);
            merge_slot(h, x4.w, n4.w, w4.w, t4.w, xo.w, no.w);
            *reinterpret_cast<float4 *>(orow + v) = xo;
            *reinterpret_cast<int4 *>(nrow + v) = no;
        }
    } else {
        for (int v = lane; v < V; v += kWave) {
            float x;
            int n;
            merge_slot(h, ls[v], ln[v], dw[v], dt[v], x, n);
            orow[v] = x;
            nrow[v] = n;
        }
    }
}

template <int HPB>
static hipError_t launch_hpb(const DevTrie &t, const int32_t *states, int64_t B, float *scores,
                             int32_t *next, hipStream_t stream, bool vec) {
    const int64_t blocks = (B + HPB - 1) / HPB;
    const size_t lds = size_t(HPB) * 2 * size_t(t.vocab_size) * sizeof(float);
    if (vec)
        hipLaunchKernelGGL((advance_kernel<HPB, true>), dim3(unsigned(blocks)), dim3(HPB * kWave), lds, stream,
                           t, states, B, scores, next);
    else
        hipLaunchKernelGGL((advance_kernel<HPB, false>), dim3(unsigned(blocks)), dim3(HPB * kWave), lds, stream,
                           t, states, B, scores, next);
    return hipGetLastError();
}

// Wavefronts per workgroup: as many rows as fit in 32 KiB of LDS, at most 4.
int advance_rows_per_block(int V) {
    const size_t row = size_t(V) * 8;
    if (4 * row <= 32768) return 4;
    if (2 * row <= 32768) return 2;
    return 1;
}

hipError_t launch_advance(const DevTrie &t, const int32_t *states, int64_t B, float *scores, int32_t *next,
                          hipStream_t stream) {
    const bool vec = (t.vocab_size % 4 == 0) && (reinterpret_cast<uintptr_t>(scores) % 16 == 0) &&
                     (reinterpret_cast<uintptr_t>(next) % 16 == 0);
    switch (advance_rows_per_block(t.vocab_size)) {
        case 4: return launch_hpb<4>(t, states, B, scores, next, stream, vec);
        case 2: return launch_hpb<2>(t, states, B, scores, next, stream, vec);
        default: return launch_hpb<1>(t, states, B, scores, next, stream, vec);
    }
}

}  // namespace ngpu
