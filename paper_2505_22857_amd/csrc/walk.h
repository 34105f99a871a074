// Device-side backoff walk shared by the advance and fused-step kernels.
//
// One wavefront (64 lanes) owns one hypothesis and a V-wide row in LDS
// (ls[v] = score or raw dense weight, ln[v] = next state with flag bits); the
// fused kernels can also split a hypothesis over W wavefronts, each owning
// every W-th stripe of 256 tokens of the row (walk_record<W>).
// The walk of state s:
//   1. its chain record (head + one entry per state of order >= 2 on its
//      backoff chain) arrives in one vector load: lane 0 reads the head, lane
//      j the entry of level j - 1.  The record's length follows from s alone
//      (its order), so nothing waits on the head to fetch the levels.
//   2. the dense row of the order-1 ancestor (which already folds in the
//      empty context) is copied global -> LDS by the load unit into the row
//      (when the caller already knows the dense row from the chain head, before
//      the record load: walk_into_lds_dense_first).
//   3. the sparse levels are applied bottom-up (order 2 first, the query
//      state's order last), each overwriting the slots of its tokens with the
//      final score and the next state marked kFinal, so the highest order that
//      holds a token wins, as in Algorithm 1.  Arcs below the highest order
//      are 8-byte records {token, weight} whose next state is their index plus
//      a constant; those of the highest order carry it, in 12 bytes.  Up to
//      four 64-arc stripes of a level are loaded (one load per lane each)
//      before any of them is written.  When the W wavefronts of a hypothesis
//      own one 256-token stripe each, every wavefront loads only the arcs of
//      its stripe, a contiguous part of each level (arcs are sorted by token).
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

#include <type_traits>

#include "trie.h"

namespace ngpu {

constexpr int kWave = 64;
constexpr int32_t kFinal = 0x40000000;         // ln bit: slot written by a sparse level
constexpr int32_t kStateMask = 0x3fffffff;
static_assert(int64_t(kStateMask) + 1 == NGPU_LM_MAX_STATES, "state ids fit the bits below the flags");

// Waits until every global -> LDS copy (and every other vector memory access)
// of this wavefront has completed.  The compiler does not reliably order LDS
// reads after those copies by itself, so every reader of copied data waits
// here first; the memory clobber keeps the compiler from moving any memory
// access across the wait.
__device__ __forceinline__ void wait_lds_copies() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// The same wait when exactly one vector memory instruction was issued after
// the last copy (vector memory loads complete in order): that one may stay in
// flight.  Callers put a compiler barrier (memory_order_point) between the
// copies and that instruction, so the compiler cannot move it above them.
__device__ __forceinline__ void wait_lds_copies_but_last() { asm volatile("s_waitcnt vmcnt(1)" ::: "memory"); }
__device__ __forceinline__ void memory_order_point() { asm volatile("" ::: "memory"); }

// vmcnt(0) as an instruction the compiler's wait insertion accounts for
// (expcnt and lgkmcnt at their maximum: no wait on them); for waits on
// loads into registers, whose data dependences already order their users.
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x0f70); }

typedef __attribute__((address_space(1))) const void global_cptr;
typedef __attribute__((address_space(3))) void lds_ptr;

// Kernel arguments are otherwise loaded (scalar loads) where first used, each
// waited for before the next is issued; in a latency-bound launch that puts
// several scalar memory round trips before the first state load.  Passing
// them to empty asm statements at the kernel's start issues all their loads at
// once, with one wait; later reads reuse the values (kernel arguments are
// constant) or hit the scalar cache.  The asm statements count as memory
// accesses, so uniform loads from global memory after them are vector loads.
// Used by the small-batch kernels only: kernels with a loop over hypotheses or
// frames would hold the values in scalar registers throughout and spill.
template <class T>
__device__ __forceinline__ void load_arg(const T &v) {
    asm volatile("" ::"s"(v));
}
template <class... T>
__device__ __forceinline__ void load_args(const T &...v) {
    (load_arg(v), ...);
}

__device__ __forceinline__ void load_trie_args(const DevTrie &t) {
    load_args(t.chain, t.dense_w, t.dense_to, t.arcs, t.top_arcs, t.status, t.num_states, t.vocab_size, t.top_begin,
              t.to_delta);
    load_args(t.first[1], t.first[2], t.first[3], t.first[4], t.first[5], t.first[6], t.first[7], t.first[8],
              t.first[9]);
    load_args(t.off_order[0], t.off_order[1], t.off_order[2], t.off_order[3], t.off_order[4], t.off_order[5],
              t.off_order[6], t.off_order[7], t.off_order[8], t.off_order[9]);
    static_assert(NGPU_LM_MAX_ORDER == 10, "the chain tables above have NGPU_LM_MAX_ORDER entries");
}

// LDS row length: V rounded up to whole 256-token copy stripes.
__host__ __device__ inline int lds_row(int V) { return (V + 255) & ~255; }

// Chain record address of state s (s in [0, num_states), one per lane) and its
// number of levels.
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

// The per-order tables of chain_record spread over the lanes of a wavefront,
// built once per kernel: lane j (1 <= j < NGPU_LM_MAX_ORDER) holds first[j],
// every other lane a bound no state reaches, and lane j holds base[j] with
// record(s) = chain + base[k] + 16 max(k, 1) s for a state s of order k.  A
// uniform state's order is then one compare, a ballot and a popcount, and its
// base one pair of readlanes: no memory access and no scalar registers held
// across the loops of the kernels (the tables from the kernel arguments would
// be loaded again at every use there).
struct ChainIndex {
    int32_t first;
    uint64_t base;
};

// (The empty asm keeps the compiler from moving the construction down to the
// first lookup, after the state load it is meant to overlap.)
__device__ __forceinline__ ChainIndex chain_index(const DevTrie &t, int lane) {
    ChainIndex ci{0x7fffffff, 0};
#pragma unroll
    for (int j = 0; j < NGPU_LM_MAX_ORDER; ++j) {
        if (lane == j) {
            const int32_t f = j == 0 ? 0 : t.first[j];
            ci.first = j == 0 ? 0x7fffffff : f;
            ci.base = t.off_order[j] - uint64_t(16 * (j > 0 ? j : 1)) * uint64_t(f);
        }
    }
    asm volatile("" ::"v"(ci.first), "v"(ci.base));
    return ci;
}

// How a kernel finds the record of a uniform state (every lane of the
// wavefront active):
//  - KernargTables: the tables from the kernel arguments where used (the
//    compiler turns the selection into one load from a selected address,
//    after the state has arrived); the choice of the grouped advance, which
//    walks many hypotheses per wavefront;
//  - ChainIndex (above), built where the kernel starts: its order from one
//    compare, a ballot and a popcount, its base from two readlanes.  Holding
//    the tables in scalar registers instead costs about a hundred scalar
//    instructions per lookup (a select per order for the order, the offset
//    and the first id), and makes the decode spill.
struct KernargTables {};

__device__ __forceinline__ const unsigned char *chain_record(const DevTrie &t, KernargTables, int s, int &nlev) {
    return chain_record(t, s, nlev);
}

__device__ __forceinline__ const unsigned char *chain_record(const DevTrie &t, const ChainIndex &ci, int s,
                                                            int &nlev) {
    const int k = __builtin_popcountll(__ballot(s >= ci.first));
    const uint64_t base = (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(ci.base >> 32), k))) << 32) |
                          uint32_t(__builtin_amdgcn_readlane(int(uint32_t(ci.base)), k));
    nlev = k > 1 ? k - 1 : 0;
    return t.chain + base + uint64_t(s) * uint64_t(16 * (k > 0 ? k : 1));
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

// Token stripes: tokens [256c, 256c + 256) form stripe c.  When W wavefronts
// share one hypothesis, wavefront w owns the stripes c with c % W == w: it
// alone copies, writes and reads their LDS slots, so the wavefronts of a
// hypothesis never touch each other's slots.  W = 1: one wavefront owns all.
constexpr int kStripe = 256;

template <int W>
__device__ __forceinline__ bool owns_token(int tok, int wave) {
    return W == 1 || ((tok >> 8) & (W - 1)) == wave;
}

// Arc range of record entry j for wavefront `wave` of W: the whole level, or,
// when SPLIT (the wavefronts own one 256-token stripe each), the part of it
// whose tokens fall in the wavefront's stripe, from the level's split counts.
template <int W, bool SPLIT, bool HALVES = false>
__device__ __forceinline__ void level_bounds(const int4 &rec, int j, int wave, int &a0, int &end) {
    a0 = __builtin_amdgcn_readlane(rec.x, j);
    end = __builtin_amdgcn_readlane(rec.y, j);
    if (HALVES) {   // wavefront `wave` owns tokens [512 wave, 512 wave + 512)
        const int c2 = int((unsigned(__builtin_amdgcn_readlane(rec.w, j)) >> 9) & 0x3ffu);
        if (wave == 0)
            end = a0 + c2;
        else
            a0 += c2;
    } else if (SPLIT && W > 1) {
        const unsigned sp = unsigned(__builtin_amdgcn_readlane(rec.w, j));
        const int n = end - a0;
        const int c1 = int(sp & 0x1ffu), c2 = int((sp >> 9) & 0x3ffu), c3 = int((sp >> 19) & 0x3ffu);
        const int lo = wave == 0 ? 0 : (wave == 1 ? c1 : (wave == 2 ? c2 : c3));
        const int hi = wave == W - 1 ? n : (wave == 0 ? c1 : (wave == 1 ? c2 : c3));
        end = a0 + hi;
        a0 += lo;
    }
}

// Word 3 of a raw (unformatted, unswizzled) buffer resource on gfx9-family
// chips: 32-bit data format; reads past the resource's byte range return 0.
constexpr int kBufferConfig = 0x00020000;

// Issues the load of state s's chain record (s uniform and valid); nlev is its
// number of levels.  The record is consumed by walk_record().
template <class Index>
__device__ __forceinline__ int4 fetch_record(const DevTrie &t, const Index &ci, int s, int lane, int &nlev) {
    const unsigned char *rp = chain_record(t, ci, s, nlev);
    return load_record(rp, nlev, lane);
}

// n words from src (global) into dst (LDS), the owned stripes only; dst padded
// to whole stripes.
template <int W>
__device__ __forceinline__ void copy_stripes_dword(const void *src, void *dst, int n, int wave, int lane) {
    if (W == 1) {
        copy_to_lds_dword(src, dst, n, lane);
        return;
    }
    const uint32_t *s = static_cast<const uint32_t *>(src);
    uint32_t *d = static_cast<uint32_t *>(dst);
    for (int c = kStripe * wave; c < n; c += kStripe * W)
        copy_to_lds_dword(s + c, d + c, n - c < kStripe ? n - c : kStripe, lane);
}

// Tokens [512 part, 512 part + 512) of dense row `row` into (ls, ln), which
// hold that half only (slot = token - 512 part; V a multiple of 4).
__device__ __forceinline__ void dense_half_to_lds(const DevTrie &t, int row, float *ls, int *ln, int part,
                                                  int lane) {
    const int V = t.vocab_size;
    const float *dw = t.dense_w + size_t(row) * V;
    const int32_t *dt = t.dense_to + size_t(row) * V;
    const int c0 = 2 * kStripe * part;
    for (int c = c0; c < V && c < c0 + 2 * kStripe; c += kStripe) {
        const int n = V - c < kStripe ? V - c : kStripe;
        copy_to_lds_x4(dw + c, ls + (c - c0), n, lane);
        copy_to_lds_x4(dt + c, ln + (c - c0), n, lane);
    }
}

template <int W>
__device__ __forceinline__ void dense_stripes_to_lds(const DevTrie &t, int row, float *ls, int *ln, int wave,
                                                     int lane) {
    if (W == 1) {
        dense_to_lds(t, row, ls, ln, lane);
        return;
    }
    const int V = t.vocab_size;
    const float *dw = t.dense_w + size_t(row) * V;
    const int32_t *dt = t.dense_to + size_t(row) * V;
    for (int c = kStripe * wave; c < V; c += kStripe * W) {
        const int n = V - c < kStripe ? V - c : kStripe;
        if ((V & 3) == 0) {
            copy_to_lds_x4(dw + c, ls + c, n, lane);
            copy_to_lds_x4(dt + c, ln + c, n, lane);
        } else {
            copy_to_lds_dword(dw + c, ls + c, n, lane);
            copy_to_lds_dword(dt + c, ln + c, n, lane);
        }
    }
}

__device__ __forceinline__ int next_of(const Arc &, int a, int to_delta) { return a + to_delta; }
__device__ __forceinline__ int next_of(const TopArc &r, int, int) { return r.to; }

// Arcs [a0, end) of one level, all of one order, applied to (ls, ln) with
// accumulator acc: four 64-arc stripes per round trip.  TOP: the level's arcs
// are of the highest order, records with their next state (top_arcs); below
// it an arc's next state is its index plus to_delta.
template <int W, bool HALVES, bool TOP>
__device__ __forceinline__ void apply_level(const DevTrie &t, int a0, int end, float acc, float *ls, int *ln,
                                            int lane, int wave) {
    typedef typename std::conditional<TOP, TopArc, Arc>::type Rec;
    const Rec *recs = TOP ? reinterpret_cast<const Rec *>(t.top_arcs) : reinterpret_cast<const Rec *>(t.arcs);
    const int first = TOP ? t.top_begin : 0;   // index of recs[0]
    for (; a0 < end; a0 += 4 * kWave) {
        // (loaded straight into the array, with no copy in the branch that
        // would have to wait for the load)
        Rec r[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int a = a0 + u * kWave + lane;
            if (a < end) r[u] = recs[a - first];
        }
        // one wait the compiler sees for all the loads: otherwise, since the
        // writes below may be skipped, it keeps them pending across the loop
        // and waits before each load of the next chunk
        wait_loads();
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int a = a0 + u * kWave + lane;
            if (a < end && (HALVES || owns_token<W>(r[u].tok, wave))) {
                const int slot = HALVES ? r[u].tok - 2 * kStripe * wave : r[u].tok;
                ls[slot] = acc + r[u].w;
                ln[slot] = next_of(r[u], a, t.to_delta) | kFinal;
            }
        }
    }
}

// The walk of a fetched record into (ls, ln), the stripes of wavefront `wave`
// of W (SPLIT: each wavefront owns exactly one stripe, and loads only its part
// of each level; HALVES: two wavefronts, each owning one 512-token half).
// When pf_src is given, pf_n words from it are also copied into pf_dst (the
// owned stripes) once the record is in (a prefetch that rides along with the
// dense row and the arcs).  DENSE_ISSUED: the caller already issued the copy
// of the dense row (before any arc load, which orders the arcs' LDS writes
// after it).
template <int W = 1, bool SPLIT = false, bool DENSE_ISSUED = false, bool HALVES = false>
__device__ __forceinline__ ChainHead walk_record(const DevTrie &t, const int4 &rec, int nlev, float *ls, int *ln,
                                                 int lane, int wave = 0, const float *pf_src = nullptr,
                                                 float *pf_dst = nullptr, int pf_n = 0) {
    const ChainHead h = head_of(rec);
    if (!DENSE_ISSUED) {
        if (HALVES)
            dense_half_to_lds(t, h.dense_row, ls, ln, wave, lane);
        else
            dense_stripes_to_lds<W>(t, h.dense_row, ls, ln, wave, lane);
    }
    if (pf_src) copy_stripes_dword<W>(pf_src, pf_dst, pf_n, wave, lane);
    for (int j = nlev; j >= 1; --j) {
        int a0, end;
        level_bounds<W, SPLIT, HALVES>(rec, j, wave, a0, end);
        const float acc = __int_as_float(__builtin_amdgcn_readlane(rec.z, j));
        if (a0 >= t.top_begin)   // uniform: a level holds arcs of one order
            apply_level<W, HALVES, true>(t, a0, end, acc, ls, ln, lane, wave);
        else
            apply_level<W, HALVES, false>(t, a0, end, acc, ls, ln, lane, wave);
    }
    wait_lds_copies();
    return h;
}

// The walk of uniform state s into (ls, ln).
template <class Index>
__device__ __forceinline__ ChainHead walk_into_lds(const DevTrie &t, const Index &ci, int s, float *ls, int *ln,
                                                   int lane) {
    int nlev;
    const int4 rec = fetch_record(t, ci, s, lane, nlev);
    return walk_record(t, rec, nlev, ls, ln, lane);
}

// The same walk when the state's dense row is already known (from its chain
// head): the row's copy into LDS goes out before the record load, so the two
// overlap instead of the copy waiting for the record.
template <class Index>
__device__ __forceinline__ ChainHead walk_into_lds_dense_first(const DevTrie &t, const Index &ci, int s,
                                                               int dense_row, float *ls, int *ln, int lane) {
    dense_to_lds(t, dense_row, ls, ln, lane);
    int nlev;
    const int4 rec = fetch_record(t, ci, s, lane, nlev);
    return walk_record<1, false, true>(t, rec, nlev, ls, ln, lane);
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

// One step of the wave maximum: each lane takes the larger of its value and
// the value DPP control CTRL moves into it (lanes with no source, or outside
// ROW_MASK, see 0, which never wins since the values are unsigned).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ unsigned max_step(unsigned k) {
    const unsigned o = unsigned(__builtin_amdgcn_update_dpp(0, int(k), CTRL, ROW_MASK, 0xf, true));
    return o > k ? o : k;
}

// Wave-wide maximum of an unsigned value, uniform in every lane.  An inclusive
// scan within each row of 16 lanes (row_shr 1, 2, 4, 8), then row 15
// broadcast into rows 1 and 3 and row 31 into rows 2 and 3, leaves the
// maximum in lane 63.
__device__ __forceinline__ unsigned wave_max_u32(unsigned k) {
    k = max_step<0x111, 0xf>(k);
    k = max_step<0x112, 0xf>(k);
    k = max_step<0x114, 0xf>(k);
    k = max_step<0x118, 0xf>(k);
    k = max_step<0x142, 0xa>(k);
    k = max_step<0x143, 0xc>(k);
    return unsigned(__builtin_amdgcn_readlane(int(k), kWave - 1));
}

// Order-preserving map of a float to an unsigned value; -0 counts as +0 so
// that equal values tie exactly as under a '>' comparison.
__device__ __forceinline__ unsigned value_key(float x) {
    if (x == 0.0f) x = 0.0f;
    const unsigned u = __float_as_uint(x);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Argmax key: larger value first, then smaller index (value key in the high
// word, ~index in the low word).
__device__ __forceinline__ unsigned long long argmax_key(float x, int idx) {
    return ((unsigned long long)value_key(x) << 32) | (unsigned)(~(unsigned)idx);
}

__device__ __forceinline__ int argmax_index(unsigned long long key) { return (int)(~(unsigned)(key & 0xffffffffu)); }

// The value an argmax key was made from (-0 comes back as +0).
__device__ __forceinline__ float key_value(unsigned long long key) {
    unsigned u = unsigned(key >> 32);
    u = (u & 0x80000000u) ? (u & 0x7fffffffu) : ~u;
    return __uint_as_float(u);
}

// Wave maximum of the lanes' argmax keys (value bx, index bi), uniform: the
// largest value in one 32-bit pass, then the smallest index among the lanes
// holding it in a second (a lane not holding it offers 0, below every ~index).
__device__ __forceinline__ unsigned long long wave_argmax_key(float bx, int bi) {
    const unsigned vk = value_key(bx);
    const unsigned m = wave_max_u32(vk);
    const unsigned ik = wave_max_u32(vk == m ? ~(unsigned)bi : 0u);
    return ((unsigned long long)m << 32) | ik;
}

// Per-lane running argmax over indices taken in ascending order: a strictly
// larger value replaces the best, so the lane keeps its lowest index among
// equal values.  kNone marks a lane that has seen nothing above -inf.
constexpr int kNone = 0x7fffffff;

__device__ __forceinline__ void take_max(float f, int v, float &bx, int &bi) {
    if (f > bx) {
        bx = f;
        bi = v;
    }
}

// Wave argmax of the lanes' (bx, bi): the lowest index among the largest
// values, and that value.  kNone when every value was -inf.
__device__ __forceinline__ int wave_argmax(float bx, int bi, float &best) {
    const unsigned long long k = wave_argmax_key(bx, bi);
    best = key_value(k);
    return argmax_index(k);
}

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

}  // namespace ngpu
