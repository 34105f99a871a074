// Device-side backoff walk shared by the advance and fused-step kernels.
//
// One wavefront (64 lanes) owns one hypothesis and a V-wide row in LDS
// (ls[v] = score or raw dense weight, ln[v] = next state with flag bits).
// The walk of state s:
//   1. its chain record (head + one entry per state of order >= 2 on its
//      backoff chain) arrives in one vector load: lane 0 reads the head, lane
//      j the entry of level j - 1.  The record's length follows from s alone
//      (its order), so nothing waits on the head to fetch the levels.
//   2. the dense row of the order-1 ancestor (which already folds in the
//      empty context) is copied global -> LDS by the load unit into the row,
//      together with the first stripe of sparse arcs.
//   3. the sparse levels are applied bottom-up (order 2 first, the query
//      state's order last), each overwriting the slots of its tokens with the
//      final score and the next state marked kFinal, so the highest order that
//      holds a token wins, as in Algorithm 1.
//   4. the reader turns each slot into (score, next): kFinal slots as they are,
//      raw dense slots as acc + weight with acc = acc0 where the dense entry is
//      flagged as backed off to the empty context, else acc1.
// Races: tokens within a level are distinct, so lanes never write the same
// slot in one level; LDS operations of one wavefront complete in program
// order.  A global -> LDS copy lands asynchronously: the sparse writes wait
// for their own arc loads, issued after the copy (vector memory loads complete
// in order), and every reader of copied data first calls wait_lds_copies().
#pragma once

#include <hip/hip_runtime.h>

#include "trie.h"

namespace ngpu {

constexpr int kWave = 64;
constexpr int kArcUnroll = 4;                  // arc stripes of 64 lanes loaded before their LDS writes
constexpr int32_t kFinal = 0x40000000;         // ln bit: slot written by a sparse level
constexpr int32_t kStateMask = 0x3fffffff;

// Waits until every global -> LDS copy (and every other vector memory access)
// of this wavefront has completed.  The compiler does not reliably order LDS
// reads after those copies by itself, so every reader of copied data waits
// here first; the memory clobber keeps the compiler from moving any memory
// access across the wait.
__device__ __forceinline__ void wait_lds_copies() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

typedef __attribute__((address_space(1))) const void global_cptr;
typedef __attribute__((address_space(3))) void lds_ptr;

// LDS row length: V rounded up to whole 256-token copy stripes.
__host__ __device__ inline int lds_row(int V) { return (V + 255) & ~255; }

// Chain record address of state s (s in [0, num_states)) and its number of levels.
__device__ __forceinline__ const unsigned char *chain_record(const DevTrie &t, int s, int &nlev) {
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
    nlev = k > 1 ? k - 1 : 0;
    return t.chain + off + size_t(s - fk) * 16u * size_t(k > 0 ? k : 1);
}

__device__ __forceinline__ int chain_group(const ChainHead &h) { return h.nlev_group >> 16; }

// Lane 0: the head; lane j in [1, nlev]: level j - 1; other lanes: zeros.
__device__ __forceinline__ int4 load_record(const unsigned char *rp, int nlev, int lane) {
    int4 r = make_int4(0, 0, 0, 0);
    if (lane <= nlev) r = *reinterpret_cast<const int4 *>(rp + 16 * lane);
    return r;
}

__device__ __forceinline__ ChainHead head_of(const int4 &r) {
    ChainHead h;
    h.dense_row = __builtin_amdgcn_readlane(r.x, 0);
    h.acc1 = __int_as_float(__builtin_amdgcn_readlane(r.y, 0));
    h.acc0 = __int_as_float(__builtin_amdgcn_readlane(r.z, 0));
    h.nlev_group = __builtin_amdgcn_readlane(r.w, 0);
    return h;
}

// Copies n contiguous 32-bit words from global src to LDS dst (uniform
// pointers) with the load unit; lanes past n re-read the last word and write
// into dst's padding, which must extend to a multiple of 64 words.
__device__ __forceinline__ void copy_to_lds_dword(const void *src, void *dst, int n, int lane) {
    const uint32_t *s = static_cast<const uint32_t *>(src);
    for (int c = 0; c < n; c += kWave) {
        const int i = c + lane < n ? c + lane : n - 1;
        __builtin_amdgcn_global_load_lds((global_cptr *)(s + i), (lds_ptr *)(static_cast<uint32_t *>(dst) + c), 4,
                                         0, 0);
    }
}

// Same for n a multiple of 4 and 16-byte aligned src and dst, 16 bytes per lane;
// dst padding up to a multiple of 256 words.
__device__ __forceinline__ void copy_to_lds_x4(const void *src, void *dst, int n, int lane) {
    const uint32_t *s = static_cast<const uint32_t *>(src);
    for (int c = 0; c < n; c += 4 * kWave) {
        const int i = c + 4 * lane < n ? c + 4 * lane : n - 4;
        __builtin_amdgcn_global_load_lds((global_cptr *)(s + i), (lds_ptr *)(static_cast<uint32_t *>(dst) + c), 16,
                                         0, 0);
    }
}

// Dense row `row` into (ls, ln) as raw (weight, flagged state).
__device__ __forceinline__ void dense_to_lds(const DevTrie &t, int row, float *ls, int *ln, int lane) {
    const int V = t.vocab_size;
    const float *dw = t.dense_w + size_t(row) * V;
    const int32_t *dt = t.dense_to + size_t(row) * V;
    if ((V & 3) == 0) {   // rows of a 256-byte aligned section are 16-byte aligned
        copy_to_lds_x4(dw, ls, V, lane);
        copy_to_lds_x4(dt, ln, V, lane);
    } else {
        copy_to_lds_dword(dw, ls, V, lane);
        copy_to_lds_dword(dt, ln, V, lane);
    }
}

// One stripe group of a level's arcs: loads for arcs a0 + lane + 64u, u < kArcUnroll.
struct ArcStripe {
    int tok[kArcUnroll];
    int to[kArcUnroll];
    float w[kArcUnroll];
};

__device__ __forceinline__ void load_stripe(const DevTrie &t, int a0, int end, int lane, ArcStripe &st) {
#pragma unroll
    for (int u = 0; u < kArcUnroll; ++u) {
        const int a = a0 + u * kWave + lane;
        st.tok[u] = -1;
        if (a < end) {
            st.tok[u] = t.arc_tok[a];
            st.w[u] = t.arc_w[a];
            st.to[u] = t.arc_to[a];
        }
    }
}

__device__ __forceinline__ void store_stripe(const ArcStripe &st, float acc, float *ls, int *ln) {
#pragma unroll
    for (int u = 0; u < kArcUnroll; ++u) {
        if (st.tok[u] >= 0) {
            ls[st.tok[u]] = acc + st.w[u];
            ln[st.tok[u]] = st.to[u] | kFinal;
        }
    }
}

// The walk of uniform state s into (ls, ln).  When pf_src is given, pf_n words
// from it are also copied into pf_dst once the record is in (a prefetch that
// rides along with the dense row and the arcs).
__device__ __forceinline__ ChainHead walk_into_lds(const DevTrie &t, int s, float *ls, int *ln, int lane,
                                                   const float *pf_src = nullptr, float *pf_dst = nullptr,
                                                   int pf_n = 0) {
    int nlev;
    const unsigned char *rp = chain_record(t, s, nlev);
    const int4 rec = load_record(rp, nlev, lane);
    const ChainHead h = head_of(rec);
    dense_to_lds(t, h.dense_row, ls, ln, lane);
    if (pf_src) copy_to_lds_dword(pf_src, pf_dst, pf_n, lane);
    // levels bottom-up: entry nlev (order 2) first, entry 1 (the query state) last
    for (int j = nlev; j >= 1; --j) {
        const int begin = __builtin_amdgcn_readlane(rec.x, j);
        const int end = __builtin_amdgcn_readlane(rec.y, j);
        const float acc = __int_as_float(__builtin_amdgcn_readlane(rec.z, j));
        for (int a0 = begin; a0 < end; a0 += kWave * kArcUnroll) {
            ArcStripe st;
            load_stripe(t, a0, end, lane, st);
            store_stripe(st, acc, ls, ln);
        }
    }
    // Every copy into LDS has landed from here on.  Waiting once here also keeps
    // the readers' loops free of waits: on gfx950 stores count in vmcnt too, so
    // a wait inside a loop that also stores would drain those stores each turn.
    wait_lds_copies();
    return h;
}

// Final (score, next state) of one LDS slot.
__device__ __forceinline__ void slot_value(const ChainHead &h, float x, int n, float &score, int &next) {
    if (n & kFinal) {
        score = x;
        next = n & kStateMask;
    } else {
        score = ((n & kDenseBackoff) ? h.acc0 : h.acc1) + x;
        next = n & kStateMask;
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
