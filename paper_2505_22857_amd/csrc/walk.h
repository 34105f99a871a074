// Device-side backoff walk shared by the advance and fused-step kernels.
//
// One wavefront (64 lanes) owns one hypothesis.  Its state's chain record
// (one 16-byte head plus one 16-byte entry per state of order >= 2 on the
// backoff chain) gives every sparse level's arc range and accumulator at
// once, so the only dependent loads are state -> chain record -> arcs.  The
// sparse levels are scattered, highest order first (Algorithm 1), into the
// wavefront's V-wide LDS row (ln[v] = next state or -1 while unset, ls[v] =
// score), with all arc loads of a stripe issued before any LDS access.  The
// order-1 ancestor's dense row, which already folds in the empty context,
// supplies every slot left unset; it is merged by whoever reads the LDS row.
//
// Races: within a level the tokens are distinct, so lanes never write the same
// slot; across levels the LDS operations of one wavefront complete in program
// order, so a later (lower-order) level sees every slot an earlier level set.
#pragma once

#include <hip/hip_runtime.h>

#include "trie.h"

namespace ngpu {

constexpr int kWave = 64;
constexpr int kArcUnroll = 4;   // arc stripes of 64 lanes loaded before the LDS scatter

// Chain record of state s (s in [0, num_states)); per-lane or uniform.
__device__ __forceinline__ const unsigned char *chain_record(const DevTrie &t, int s) {
    int k = 0, fk = 0;
    uint64_t off = t.off_order[0];
#pragma unroll
    for (int j = 1; j < NGPU_LM_MAX_ORDER; ++j) {
        if (s >= t.first[j]) {   // first[] ascends; entries past the last order equal S
            k = j;
            fk = t.first[j];
            off = t.off_order[j];
        }
    }
    return t.chain + off + size_t(s - fk) * 16u * size_t(k > 0 ? k : 1);
}

__device__ __forceinline__ int chain_levels(const ChainHead &h) { return h.nlev_group & 0xffff; }
__device__ __forceinline__ int chain_group(const ChainHead &h) { return h.nlev_group >> 16; }

// Scatters the sparse levels of a chain record (uniform rp) into (ls, ln).
__device__ __forceinline__ void scatter_levels(const DevTrie &t, const unsigned char *rp, int nlev, float *ls,
                                               int *ln, int lane) {
    const int V = t.vocab_size;
    const ChainLevel *lev = reinterpret_cast<const ChainLevel *>(rp + sizeof(ChainHead));
    for (int v = lane; v < V; v += kWave) ln[v] = -1;
    for (int j = 0; j < nlev; ++j) {
        const ChainLevel L = lev[j];
        for (int a0 = L.begin; a0 < L.end; a0 += kWave * kArcUnroll) {
            int tok[kArcUnroll], to[kArcUnroll];
            float w[kArcUnroll];
#pragma unroll
            for (int u = 0; u < kArcUnroll; ++u) {
                const int a = a0 + u * kWave + lane;
                tok[u] = -1;
                if (a < L.end) {
                    tok[u] = t.arc_tok[a];
                    w[u] = t.arc_w[a];
                    to[u] = t.arc_to[a];
                }
            }
#pragma unroll
            for (int u = 0; u < kArcUnroll; ++u) {
                if (tok[u] >= 0 && ln[tok[u]] < 0) {
                    ls[tok[u]] = L.acc + w[u];
                    ln[tok[u]] = to[u];
                }
            }
        }
    }
}

// Walks uniform state s into (ls, ln); returns the chain head.
__device__ __forceinline__ ChainHead walk_into_lds(const DevTrie &t, int s, float *ls, int *ln, int lane) {
    const unsigned char *rp = chain_record(t, s);
    const ChainHead head = *reinterpret_cast<const ChainHead *>(rp);
    scatter_levels(t, rp, chain_levels(head), ls, ln, lane);
    return head;
}

// Final value of one token: the LDS slot if a sparse level set it, else the
// dense row entry with the accumulator its flag selects.
__device__ __forceinline__ void merge_slot(const ChainHead &h, float lsv, int lnv, float dw, int dt, float &x, int &n) {
    if (lnv >= 0) {
        x = lsv;
        n = lnv;
    } else {
        x = ((dt & kDenseBackoff) ? h.acc0 : h.acc1) + dw;
        n = dt & 0x7fffffff;
    }
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
