// Device-side backoff walk shared by the advance and fused-step kernels.
//
// One wavefront (64 lanes) owns one hypothesis and a V-wide row in LDS:
// ln[v] = next state (-1 while no level above the empty context holds v),
// ls[v] = score.  The walk visits the query state and its backoff states down
// to (not including) the empty context, highest order first (Algorithm 1):
// each level's arcs are spread over the lanes and scattered into the slots that
// are still unset, then the level's backoff weight joins the accumulator.  The
// dense empty-context row is merged afterwards by whoever reads the LDS row, so
// it is never scattered.  Within a level the tokens are distinct, so lanes never
// race on a slot; across levels the LDS operations of one wavefront complete in
// program order, so a later level sees every slot an earlier level set.
#pragma once

#include <hip/hip_runtime.h>

#include "trie.h"

namespace ngpu {

constexpr int kWave = 64;

// Walks state s into (ls, ln); returns the accumulator at the empty context.
__device__ __forceinline__ float walk_into_lds(const DevTrie &t, int s, float *ls, int *ln, int lane) {
    const int V = t.vocab_size;
    for (int v = lane; v < V; v += kWave) ln[v] = -1;
    float acc = 0.0f;
    // a state of order k reaches the empty context after k backoffs (k < N)
    for (int lvl = 0; lvl < t.max_order && s != 0; ++lvl) {
        const StateRec r = t.rec[s];
        for (int a = r.begin + lane; a < r.end; a += kWave) {
            const int tok = t.arc_tok[a];
            if (ln[tok] < 0) {
                ls[tok] = acc + t.arc_w[a];
                ln[tok] = t.arc_to[a];
            }
        }
        acc = acc + r.bw;
        s = r.bto;
    }
    return acc;
}

// Wave-wide maximum of a 64-bit key.
__device__ __forceinline__ unsigned long long wave_max_u64(unsigned long long k) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        unsigned lo = __shfl_xor((unsigned)(k & 0xffffffffu), off, kWave);
        unsigned hi = __shfl_xor((unsigned)(k >> 32), off, kWave);
        unsigned long long o = ((unsigned long long)hi << 32) | lo;
        k = o > k ? o : k;
    }
    return k;
}

// Argmax key: larger value first, then smaller index.  -0 counts as +0 so
// that equal values tie exactly as under a '>' comparison.
__device__ __forceinline__ unsigned long long argmax_key(float x, int idx) {
    if (x == 0.0f) x = 0.0f;
    unsigned u = __float_as_uint(x);
    u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((unsigned long long)u << 32) | (unsigned)(0xffffffffu - (unsigned)idx);
}

__device__ __forceinline__ int argmax_index(unsigned long long key) {
    return (int)(0xffffffffu - (unsigned)(key & 0xffffffffu));
}

}  // namespace ngpu
