// Greedy shallow fusion (Section 2.3): one step over a batch of hypotheses, and
// a whole decode over all frames of a batch of utterances in one launch.
//
// One workgroup of W wavefronts per hypothesis (W = 4 for batches up to 512,
// else 1), each wavefront owning every W-th stripe of 256 tokens.  CTC and
// transducer modes first take the plain ASR argmax over the V + 1 classes;
// when that keeps blank (or, for CTC, the previous label) the LM is not
// consulted at all and the state stays.  Otherwise the workgroup walks its
// state's backoff chain into an LDS row (the same walk as the advance kernel,
// with no HBM write of the row), merges the dense row of the order-1 ancestor,
// forms fmaf(lambda, lm[v], asr[v]) per token and takes the argmax with
// lowest-index ties: each lane keeps a running maximum over its tokens (read
// four at a time from LDS), the lanes' (value, index) pairs are reduced
// across the wavefront with DPP moves (the largest value, then the smallest
// index holding it), and the W wavefronts' winners meet as 64-bit keys
// (value, ~index) in one LDS exchange.  The winner's next state rides along with its key.  No
// MFMA: one fma and one compare per token.
//
// The decode kernel keeps each utterance's state and previous label in
// registers across frames: frame t + 1 depends on frame t only through them,
// so a single launch replaces T launches and their host round trips.
//
// AED mode (Section 2.3): class V is <eos>, whose LM score is the state's
// final weight (the </s> score, precomputed per state); <eos> keeps the state.
#include <hip/hip_runtime.h>

#include <atomic>

#include "walk.h"

namespace ngpu {

enum { kPlain = 0, kCtc = 1, kTransducer = 2, kAed = 3 };

// Words of an ASR row buffer in LDS: the V tokens rounded up to whole
// stripes, so that the 16-byte reads of the scans stay inside it.  (Blank or
// <eos>, class V, travels in a register.)
__host__ __device__ inline int asr_row_words(int V) { return lds_row(V); }

// Per-lane argmax of row[v] over the owned tokens v < V.  Lane l reads tokens
// 4l .. 4l + 3 of each owned stripe with one 16-byte LDS read, so every lane
// meets its tokens in ascending order.
template <int W>
__device__ __forceinline__ void scan_row(const float *row, int V, int wave, int lane, float &bx, int &bi) {
    const int full = V & ~(kStripe - 1);
#pragma unroll 4
    for (int c = kStripe * wave; c < full; c += kStripe * W) {
        const int v0 = c + 4 * lane;
        const f32x4 a = *reinterpret_cast<const f32x4 *>(row + v0);
#pragma unroll
        for (int j = 0; j < 4; ++j) take_max(a[j], v0 + j, bx, bi);
    }
    if (full < V && owns_token<W>(full, wave)) {
        const int v0 = full + 4 * lane;
        const f32x4 a = *reinterpret_cast<const f32x4 *>(row + v0);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (v0 + j < V) take_max(a[j], v0 + j, bx, bi);
    }
}

// Per-lane argmax of fmaf(lambda, lm[v], row[v]) over the owned tokens v < V,
// lm[v] from the walked LDS row; same reads as scan_row.
template <int W>
__device__ __forceinline__ void scan_fused(const ChainHead &h, const float *ls, const int *ln, const float *row,
                                           float lambda, int V, int wave, int lane, float &bx, int &bi) {
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
            if (!tail || v < V) take_max(f, v, bx, bi);
        }
    };
    const int full = V & ~(kStripe - 1);
#pragma unroll 4
    for (int c = kStripe * wave; c < full; c += kStripe * W) four(c + 4 * lane, false);
    if (full < V && owns_token<W>(full, wave)) four(full + 4 * lane, true);
}

// ASR row held in LDS (asr_row_words(V) words; the owned stripes are read).
template <int W>
struct LdsAsr {
    const float *row;
    __device__ __forceinline__ void argmax(int V, int wave, int lane, float &bx, int &bi) const {
        scan_row<W>(row, V, wave, lane, bx, bi);
    }
    __device__ __forceinline__ void fused(const ChainHead &h, const float *ls, const int *ln, float lambda, int V,
                                          int wave, int lane, float &bx, int &bi) const {
        scan_fused<W>(h, ls, ln, row, lambda, V, wave, lane, bx, bi);
    }
};

// ASR row held in registers, for V <= kRegTokens: lane l of wavefront w keeps
// classes 256 c + 64 j + l (j = 0 .. 3) of each owned stripe c, in ascending
// order, so each of its loads is one coalesced 256-byte read and the scans
// read the walked LDS row one word per lane (no bank conflicts).  The row is
// read through a buffer resource of V words: classes past V read as 0 without
// a branch (the scans skip them), so the loads are straight-line code and the
// compiler's waits for the chain record issued just before them can leave
// them in flight.  FULL: V = kRegTokens, every class present and nothing to
// skip (the per-class conditions would otherwise be held across the frame
// loop in scalar registers).
constexpr int kRegTokens = 1024;

template <int W, bool FULL>
struct RegAsr {
    static constexpr int kN = kRegTokens / (kWave * W);   // values per lane
    float a[kN];

    // first class of value i of this wavefront (uniform); the lane adds its index
    __device__ static __forceinline__ int base(int i, int wave) {
        return kStripe * (W * (i / 4) + (W == 1 ? 0 : wave)) + kWave * (i % 4);
    }

    // (the resource starts at this wavefront's first stripe: the range check
    // covers the lane and instruction offsets, not a scalar offset)
    __device__ __forceinline__ void load(const float *row, int V, int wave, int lane) {
        const int w0 = W == 1 ? 0 : kStripe * wave;
        const int n = V > w0 ? V - w0 : 0;
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(row + w0), short(0),
                                                                           n * int(sizeof(float)), kBufferConfig);
#pragma unroll
        for (int i = 0; i < kN; ++i)
            a[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                 r, (kStripe * W * (i / 4) + kWave * (i % 4) + lane) * int(sizeof(float)),
                                                 0, 0));
    }
    __device__ __forceinline__ void argmax(int V, int wave, int lane, float &bx, int &bi) const {
#pragma unroll
        for (int i = 0; i < kN; ++i) {
            const int v = base(i, wave) + lane;
            if (FULL || base(i, wave) + kWave <= V || v < V) take_max(a[i], v, bx, bi);
        }
    }
    __device__ __forceinline__ void fused(const ChainHead &h, const float *ls, const int *ln, float lambda, int V,
                                          int wave, int lane, float &bx, int &bi) const {
#pragma unroll
        for (int i = 0; i < kN; ++i) {
            const int b0 = base(i, wave);
            if (!FULL && b0 >= V) continue;   // uniform; the slots read below lie inside the padded row
            const int v = b0 + lane;
            float lm;
            int nx;
            slot_value(h, ls[v], ln[v], lm, nx);
            const float f = __builtin_fmaf(lambda, lm, a[i]);
            if (FULL || b0 + kWave <= V || v < V) take_max(f, v, bx, bi);
        }
    }
};

// One wavefront's copy of a compact dense row (DevTrie::dense_c), for the
// whole decode with rows in registers (W = 1): lane l keeps tokens 64 i + l,
// loaded like the ASR row (tokens past V read as 0 and are never used).
template <bool FULL>
struct CompactRow {
    float c[kRegTokens / kWave];

    __device__ __forceinline__ void load(const float *row, int V, int lane) {
        const __amdgpu_buffer_rsrc_t r =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(row), short(0), V * int(sizeof(float)), kBufferConfig);
#pragma unroll
        for (int i = 0; i < kRegTokens / kWave; ++i)
            c[i] = __builtin_bit_cast(float,
                                      __builtin_amdgcn_raw_buffer_load_b32(r, (kWave * i + lane) * int(sizeof(float)), 0, 0));
    }

    // Per-lane argmax of fmaf(lambda, lm[v], asr[v]): lm[v] from the LDS row
    // where a sparse level wrote it (kFinal in ln), else from this row: its
    // weight (the stored magnitude with the sign bit set) plus acc0 where the
    // sign bit marks a backed-off entry, acc1 otherwise.
    __device__ __forceinline__ void fused(const ChainHead &h, const float *ls, const int *ln,
                                          const RegAsr<1, FULL> &asr, float lambda, int V, int lane, float &bx,
                                          int &bi) const {
#pragma unroll
        for (int i = 0; i < kRegTokens / kWave; ++i) {
            const int b0 = kWave * i;
            if (!FULL && b0 >= V) continue;   // uniform; the slots read below lie inside the padded row
            const int v = b0 + lane;
            // (both words read unconditionally: a read inside the select
            // becomes a branch with its own wait, per token)
            const int n = ln[v];
            const float x = ls[v];
            const unsigned cb = __float_as_uint(c[i]);
            const float dense = ((cb >> 31) ? h.acc0 : h.acc1) + __uint_as_float(cb | 0x80000000u);
            const float lm = (n & kFinal) ? x : dense;
            const float f = __builtin_fmaf(lambda, lm, asr.a[i]);
            if (FULL || b0 + kWave <= V || v < V) take_max(f, v, bx, bi);
        }
    }

    // Next state of token w (uniform, w < V): the sparse level's where one
    // wrote the slot; else, for an own entry of the row when the image
    // numbers them by rank (orders >= 3), the row's first own-bigram state
    // (base) plus the number of own entries below w (one ballot per 64
    // tokens); else the unigram state first[1] + w.
    __device__ __forceinline__ int next_state(const DevTrie &t, const int *ln, int base, int w, int V,
                                              int lane) const {
        const int n = ln[w];
        if (n & kFinal) return n & kStateMask;
        const int j = w >> 6, b = w & (kWave - 1);
        int rank = 0;
        bool own = false;
#pragma unroll
        for (int i = 0; i < kRegTokens / kWave; ++i) {
            if (i > j) continue;   // uniform
            const bool mine = (FULL || kWave * i + lane < V) && !(__float_as_uint(c[i]) >> 31);
            const unsigned long long m = __ballot(mine);
            if (i < j) {
                rank += __builtin_popcountll(m);
            } else {
                rank += __builtin_popcountll(m & ((1ull << b) - 1ull));
                own = (m >> b) & 1ull;
            }
        }
        return own && t.compact_rank ? base + rank : t.first[1] + w;
    }
};

// Clears the kFinal marks of the LDS next-state row (lds_row(V) words) before
// the sparse levels write theirs: with compact rows no dense copy overwrites it.
__device__ __forceinline__ void clear_marks(int *ln, int V, int lane) {
    const i32x4 z = {0, 0, 0, 0};
    for (int c = 4 * lane; c < lds_row(V); c += 4 * kWave) *reinterpret_cast<i32x4 *>(ln + c) = z;
}

struct NoHook {
    __device__ __forceinline__ void operator()() const {}
};

// Exchange area of W wavefronts: two alternating buffers of W (key, payload)
// pairs, so one barrier per exchange suffices (a buffer is written again only
// after every wavefront has passed the next exchange's barrier).
struct Exchange {
    unsigned long long key[2][4];
    int payload[2][4];
};

// Waits until this wavefront's LDS writes are done, then for all wavefronts
// of the workgroup.  The memory clobber keeps the compiler from moving any
// memory access across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Argmax over the W wavefronts' lanes of (bx, bi): lowest index among the
// largest values.  Returns the index (kNone when every value was -inf), its
// value and the payload the winning lane passed in; all uniform.
template <int W>
__device__ __forceinline__ int group_argmax(float bx, int bi, int payload, float &best, int &win_payload,
                                            Exchange *xc, int &xi, int wave, int lane) {
    static_assert(W == 1 || W == 2 || W == 4, "the exchange area holds at most four wavefronts");
    const unsigned long long mine = argmax_key(bx, bi);
    unsigned long long k = wave_argmax_key(bx, bi);
    // the lane whose key won hands over its payload (the lowest such lane: keys are unique but for kNone)
    const unsigned long long won = __builtin_amdgcn_read_exec() & __ballot(mine == k);
    const int src = won ? int(__builtin_ctzll(won)) : 0;
    int pl = __builtin_amdgcn_readlane(payload, src);
    if (W > 1) {
        const int buf = xi & 1;
        ++xi;
        if (lane == 0) {
            xc->key[buf][wave] = k;
            xc->payload[buf][wave] = pl;
        }
        lds_barrier();
#pragma unroll
        for (int i = 0; i < W; ++i) {
            const unsigned long long o = xc->key[buf][i];
            const int op = xc->payload[buf][i];
            if (o > k) {
                k = o;
                pl = op;
            }
        }
        k = (static_cast<unsigned long long>(unsigned(__builtin_amdgcn_readfirstlane(int(unsigned(k >> 32))))) << 32) |
            unsigned(__builtin_amdgcn_readfirstlane(int(unsigned(k & 0xffffffffu))));
        pl = __builtin_amdgcn_readfirstlane(pl);
    }
    best = key_value(k);
    win_payload = pl;
    return argmax_index(k);
}

// Next state of token w in {0, 1} (stripe 0, owned by wavefront 0), shared
// with the other wavefronts.
template <int W>
__device__ __forceinline__ int first_token_state(const ChainHead &h, const float *ls, const int *ln, int w,
                                                 Exchange *xc, int &xi, int wave, int lane) {
    int ns = 0;
    if (wave == 0) {
        float lm;
        slot_value(h, ls[w], ln[w], lm, ns);
    }
    if (W > 1) {
        const int buf = xi & 1;
        ++xi;
        if (wave == 0 && lane == 0) xc->payload[buf][0] = ns;
        lds_barrier();
        ns = __builtin_amdgcn_readfirstlane(xc->payload[buf][0]);
    }
    return ns;
}

// One fused greedy step of a hypothesis held by W wavefronts.  asr: its V
// token ASR log-probabilities (LdsAsr: owned stripes landed unless
// ROW_PENDING, in which case their copy was issued just before; RegAsr);
// rowV: class V (blank, or <eos> in AED mode).  s: valid state (uniform); pv:
// previous label (CTC).  after_record runs once the chain record's load is
// issued.  Returns the label and updates s; all lanes of all W wavefronts
// return the same values.
template <int MODE, int W, bool ROW_PENDING, class Asr, class AfterRecord = NoHook, bool SPLIT = false,
          class Index = KernargTables>
__device__ __forceinline__ int greedy_step(const DevTrie &t, const Index &ci, const Asr &asr, float rowV,
                                           float lambda, int &s,
                                           int pv, float *ls, int *ln, Exchange *xc, int &xi, int wave, int lane,
                                           const float *pf_src = nullptr, float *pf_dst = nullptr, int pf_n = 0,
                                           AfterRecord after_record = {}) {
    const int V = t.vocab_size;
    const float fin = MODE == kAed ? t.final_w[s] : 0.0f;   // <eos> takes the state's final weight
    // The chain record is fetched first: in CTC and transducer modes its load
    // overlaps the plain ASR argmax, which may still find that the LM is not needed.
    int nlev;
    if (ROW_PENDING) memory_order_point();   // the ASR row's copies were issued before the record load
    const int4 rec = fetch_record(t, ci, s, lane, nlev);
    after_record();
    if (MODE == kCtc || MODE == kTransducer) {
        // the row, not the record: the record load (one instruction; after_record
        // adds none when the row is pending) stays in flight through the argmax
        if (ROW_PENDING) wait_lds_copies_but_last();
        float bx = -__builtin_inff(), av;
        int bi = kNone, unused;
        asr.argmax(V, wave, lane, bx, bi);
        int a = group_argmax<W>(bx, bi, 0, av, unused, xc, xi, wave, lane);
        if (a == kNone) a = 0;                    // every token at -inf: the first one, unless blank beats it
        if (rowV > av) a = V;                     // blank only when strictly larger (it has the highest index)
        if (a == V || (MODE == kCtc && a == pv)) {   // blank or repeat: no LM, no move
            if (pf_src) copy_stripes_dword<W>(pf_src, pf_dst, pf_n, wave, lane);
            return a;
        }
    }
    const ChainHead h = walk_record<W, SPLIT>(t, rec, nlev, ls, ln, lane, wave, pf_src, pf_dst, pf_n);
    // CTC: the previous label is no candidate; its slot reads NaN, which no
    // fused value built from it can pass under a strict '>'
    if (MODE == kCtc && pv >= 0 && pv < V && owns_token<W>(pv, wave) && lane == 0) {
        ls[pv] = __builtin_nanf("");
        ln[pv] = kFinal;
    }
    float bx = -__builtin_inff(), wv;
    int bi = kNone;
    asr.fused(h, ls, ln, lambda, V, wave, lane, bx, bi);
    // each lane's candidate next state rides along with its key (read from its own stripe)
    int cand = 0;
    if (bi != kNone) {
        float lm;
        slot_value(h, ls[bi], ln[bi], lm, cand);
    }
    int ns;
    int w = group_argmax<W>(bx, bi, cand, wv, ns, xc, xi, wave, lane);
    if (MODE == kAed && __builtin_fmaf(lambda, fin, rowV) > wv)
        return V;   // <eos> strictly above every token: the sentence ends, the state stays
    if (w == kNone) {   // every candidate at -inf: the first one
        w = (MODE == kCtc && pv == 0) ? 1 : 0;
        ns = first_token_state<W>(h, ls, ln, w, xc, xi, wave, lane);
    }
    s = ns;
    return w;
}

// The same step for the whole decode with rows in registers and compact
// dense rows (W = 1): the walk applies the sparse levels only, over cleared
// marks, and the dense row arrives in registers; the winner's next state
// follows from the compact row's rules.  Same selection as greedy_step.
template <int MODE, bool FULL, class AfterRecord>
__device__ __forceinline__ int greedy_step_compact(const DevTrie &t, const ChainIndex &ci,
                                                   const RegAsr<1, FULL> &asr, float rowV, float lambda, int &s,
                                                   int pv, float *ls, int *ln, Exchange *xc, int &xi, int lane,
                                                   AfterRecord after_record) {
    const int V = t.vocab_size;
    const float fin = MODE == kAed ? t.final_w[s] : 0.0f;
    int nlev;
    const int4 rec = fetch_record(t, ci, s, lane, nlev);
    after_record();
    if (MODE == kCtc || MODE == kTransducer) {
        float bx = -__builtin_inff(), av;
        int bi = kNone, unused;
        asr.argmax(V, 0, lane, bx, bi);
        int a = group_argmax<1>(bx, bi, 0, av, unused, xc, xi, 0, lane);
        if (a == kNone) a = 0;
        if (rowV > av) a = V;
        if (a == V || (MODE == kCtc && a == pv)) return a;
    }
    const ChainHead h = head_of(rec);
    clear_marks(ln, V, lane);
    CompactRow<FULL> row;
    row.load(t.dense_c + size_t(h.dense_row) * size_t(V), V, lane);
    const int base = t.dense_base[h.dense_row];
    walk_record<1, false, true>(t, rec, nlev, ls, ln, lane);
    if (MODE == kCtc && pv >= 0 && pv < V && lane == 0) {
        ls[pv] = __builtin_nanf("");
        ln[pv] = kFinal;
    }
    float bx = -__builtin_inff(), wv;
    int bi = kNone, unused;
    row.fused(h, ls, ln, asr, lambda, V, lane, bx, bi);
    int w = group_argmax<1>(bx, bi, 0, wv, unused, xc, xi, 0, lane);
    if (MODE == kAed && __builtin_fmaf(lambda, fin, rowV) > wv) return V;
    if (w == kNone) w = (MODE == kCtc && pv == 0) ? 1 : 0;   // every candidate at -inf: the first one
    s = row.next_state(t, ln, base, w, V, lane);
    return w;
}

// LDS of one hypothesis: the walked row (ls, ln), nrows ASR rows, the exchange area.
__host__ __device__ inline size_t hyp_lds_bytes(int V, int nrows) {
    return (2 * size_t(lds_row(V)) + size_t(nrows) * size_t(asr_row_words(V))) * sizeof(float) + sizeof(Exchange);
}

// One fused step; one hypothesis per workgroup of W wavefronts.
template <int MODE, int W, bool SPLIT = false>
__global__ __launch_bounds__(W * kWave) void fused_step_kernel(DevTrie t, const float *__restrict__ asr, int64_t B,
                                                                int64_t ld, float lambda,
                                                                int32_t *__restrict__ states,
                                                                int32_t *__restrict__ prev,
                                                                int32_t *__restrict__ tokens) {
    extern __shared__ float lds[];
    load_trie_args(t);
    load_args(asr, B, ld, lambda, states, prev, tokens);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int64_t b = blockIdx.x;
    if (b >= B) return;
    const int V = t.vocab_size;
    float *ls = lds;
    int *ln = reinterpret_cast<int *>(ls + lds_row(V));
    float *arow = reinterpret_cast<float *>(ln + lds_row(V));
    Exchange *xc = reinterpret_cast<Exchange *>(arow + asr_row_words(V));

    // the state, the previous label and blank's score go out first, then the
    // ASR row's copy into LDS, so their wait leaves the copy in flight
    const float *src = asr + b * ld;
    const int s_l = states[b];
    const int pv_l = MODE == kCtc ? prev[b] : -1;
    const float rowV_l = MODE == kPlain ? 0.0f : src[V];
    copy_stripes_dword<W>(src, arow, V, wave, lane);
    const ChainIndex ci = chain_index(t, lane);
    int s = __builtin_amdgcn_readfirstlane(s_l);
    const int pv = __builtin_amdgcn_readfirstlane(pv_l);
    const float rowV = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, rowV_l)));
    if (s < 0 || s >= t.num_states) {
        if (wave == 0 && lane == 0) {
            atomicAdd(&t.status[0], 1);
            tokens[b] = -1;
        }
        wait_lds_copies();   // no copy into LDS outlives the wavefront
        return;
    }
    int xi = 0;
    // every wavefront has read states[b] and prev[b] before the first exchange
    // barrier inside the step, and wavefront 0 writes them back after it
    const int label = greedy_step<MODE, W, true, LdsAsr<W>, NoHook, SPLIT>(
        t, ci, LdsAsr<W>{arow}, rowV, lambda, s, pv, ls, ln, xc, xi, wave, lane);
    if (wave == 0 && lane == 0) {
        tokens[b] = label;
        states[b] = s;
        if (MODE == kCtc) prev[b] = label;
    }
}

// Whole greedy decode: utterance b runs frames 0 .. len_b - 1 of
// asr[b * stride_b + t * stride_t + class]; one utterance per workgroup of W
// wavefronts.  NB: ASR row buffers in LDS (1 or 2), or 0 for rows held in
// registers (V <= kRegTokens; FULL: V = kRegTokens).
template <int MODE, int W, int NB, bool FULL = false, bool SPLIT = false, bool COMPACT = false>
__global__ __launch_bounds__(W * kWave) void fused_decode_kernel(DevTrie t, const float *__restrict__ asr, int64_t B,
                                                                  int64_t T, int64_t stride_b, int64_t stride_t,
                                                                  const int32_t *__restrict__ lengths, float lambda,
                                                                  int32_t *__restrict__ states,
                                                                  int32_t *__restrict__ prev,
                                                                  int32_t *__restrict__ labels,
                                                                  int32_t *__restrict__ label_states) {
    extern __shared__ float lds[];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int64_t b = blockIdx.x;
    if (b >= B) return;
    const int V = t.vocab_size;
    const int rowp = asr_row_words(V);
    // ASR rows: NB = 2 buffers, the next row's copy riding along with the walk
    // (while every utterance is resident at once, the latency-bound case), or
    // NB = 1 buffer, refilled once the frame has read it (when more utterances
    // than fit wait for a CU: the smaller LDS footprint lets more run at once),
    // or in registers (NB = 0), the next row loaded behind the chain record
    constexpr int kRowBufs = NB;
    RegAsr<W, FULL> cur_r;
    float *ls = lds;
    int *ln = reinterpret_cast<int *>(ls + lds_row(V));
    float *abuf = reinterpret_cast<float *>(ln + lds_row(V));
    Exchange *xc = reinterpret_cast<Exchange *>(abuf + kRowBufs * rowp);
    int32_t *lab = labels + b * T;
    int32_t *lst = label_states ? label_states + b * T : nullptr;

    int64_t len = T;
    if (lengths) {
        len = __builtin_amdgcn_readfirstlane(lengths[b]);
        len = len < 0 ? 0 : (len > T ? T : len);
    }
    int s = __builtin_amdgcn_readfirstlane(states[b]);
    if (s < 0 || s >= t.num_states) {
        if (wave == 0) {
            if (lane == 0) atomicAdd(&t.status[0], 1);
            for (int64_t f = lane; f < T; f += kWave) {
                lab[f] = -1;
                if (lst) lst[f] = -1;
            }
        }
        return;
    }
    int pv = MODE == kCtc ? __builtin_amdgcn_readfirstlane(prev[b]) : -1;
    const float *row = asr + b * stride_b;
    if (len > 0) {
        if (kRowBufs == 0)
            cur_r.load(row, V, wave, lane);
        else
            copy_stripes_dword<W>(row, abuf, V, wave, lane);
    }
    float rowV = (MODE != kPlain && len > 0) ? row[V] : 0.0f;
    int keep_lab = -1, keep_st = -1, xi = 0;
    const ChainIndex ci = chain_index(t, lane);
    for (int64_t f = 0; f < len; ++f, row += stride_t) {
        // LDS rows: frame f reads its ASR row from LDS, copied during frame
        // f - 1 (or before the loop); the walk also starts the copy of row
        // f + 1.  (The wait comes before any load of this frame is issued.)
        if (kRowBufs > 0) wait_lds_copies();
        const bool more = f + 1 < len;
        const float *pf = more ? row + stride_t : nullptr;
        const float next_v = (MODE != kPlain && more) ? row[stride_t + V] : 0.0f;
        int label;
        if constexpr (kRowBufs == 0) {
            // the last frame reloads its own row: with no branch around the
            // loads the compiler's count of loads in flight stays exact
            RegAsr<W, FULL> nxt_r;
            const float *src = more ? pf : row;
            auto load_next = [&]() { nxt_r.load(src, V, wave, lane); };
            if constexpr (COMPACT) {
                static_assert(W == 1, "compact dense rows serve one wavefront per utterance");
                label = greedy_step_compact<MODE, FULL>(t, ci, cur_r, rowV, lambda, s, pv, ls, ln, xc, xi, lane,
                                                        load_next);
            } else {
                label = greedy_step<MODE, W, false, RegAsr<W, FULL>, decltype(load_next), SPLIT>(
                    t, ci, cur_r, rowV, lambda, s, pv, ls, ln, xc, xi, wave, lane, nullptr, nullptr, 0, load_next);
            }
            cur_r = nxt_r;
        } else {
            float *cur = abuf + (kRowBufs == 2 ? (f & 1) * rowp : 0);
            float *nxt = abuf + (kRowBufs == 2 ? ((f + 1) & 1) * rowp : 0);
            label = greedy_step<MODE, W, false, LdsAsr<W>, NoHook, SPLIT>(
                t, ci, LdsAsr<W>{cur}, rowV, lambda, s, pv, ls, ln, xc, xi, wave, lane, kRowBufs == 2 ? pf : nullptr,
                nxt, V);
            // one buffer: every read of this frame's row has completed (its values
            // were consumed by the argmax), so the next row can be copied over it
            if (kRowBufs == 1 && pf) copy_stripes_dword<W>(pf, cur, V, wave, lane);
        }
        rowV = next_v;
        if (MODE == kCtc) pv = label;
        // Lane f % 64 of wavefront 0 keeps frame f's label and state; one
        // coalesced store per 64 frames, so the wait at the top of a frame
        // rarely has a store to drain.
        const int slot = int(f & (kWave - 1));
        if (lane == slot) {
            keep_lab = label;
            keep_st = s;
        }
        if (wave == 0 && (slot == kWave - 1 || f + 1 == len)) {
            const int64_t f0 = f - slot;
            if (lane <= slot) {
                lab[f0 + lane] = keep_lab;
                if (lst) lst[f0 + lane] = keep_st;
            }
        }
    }
    if (wave == 0) {
        for (int64_t f = len + lane; f < T; f += kWave) {   // frames past the utterance's end
            lab[f] = -1;
            if (lst) lst[f] = s;
        }
        // every wavefront read states[b] and prev[b] before the first exchange
        // barrier; with no frame at all the values written are the ones read
        if (lane == 0) {
            states[b] = s;
            if (MODE == kCtc) prev[b] = pv;
        }
    }
}

// The k best fused scores of one hypothesis per wavefront (beam-search
// expansion), in descending order with lowest-index ties.  After the walk,
// each lane turns its slots into (fused value, next state) in place and keeps
// its own best; a round reduces the lanes' bests to the winner (one DPP
// reduction), and only the lane that held it marks the slot taken (bit 31 of
// its next state), writes the outputs and rescans its own tokens.  Cost:
// V / 64 per lane once, then k rounds of one reduction and one lane's rescan.
__global__ __launch_bounds__(kWave) void fused_topk_kernel(DevTrie t, const float *__restrict__ asr, int64_t B,
                                                           int64_t ld, float lambda, int k,
                                                           const int32_t *__restrict__ states,
                                                           int32_t *__restrict__ tokens, float *__restrict__ scores,
                                                           int32_t *__restrict__ next) {
    extern __shared__ float lds[];
    load_trie_args(t);
    load_args(asr, B, ld, lambda, k, states, tokens, scores, next);
    const int lane = threadIdx.x;
    const int64_t b = blockIdx.x;
    if (b >= B) return;
    const int V = t.vocab_size;
    float *ls = lds;
    int *ln = reinterpret_cast<int *>(ls + lds_row(V));
    float *arow = reinterpret_cast<float *>(ln + lds_row(V));
    int32_t *otok = tokens + b * k;
    float *osc = scores + b * k;
    int32_t *onx = next + b * k;
    const int s_l = states[b];   // issued before the row copy, so its wait leaves the copy in flight
    copy_to_lds_dword(asr + b * ld, arow, V, lane);
    const ChainIndex ci = chain_index(t, lane);
    const int s = __builtin_amdgcn_readfirstlane(s_l);
    if (s < 0 || s >= t.num_states) {
        if (lane == 0) atomicAdd(&t.status[0], 1);
        for (int j = lane; j < k; j += kWave) {
            otok[j] = -1;
            osc[j] = NAN;
            onx[j] = -1;
        }
        wait_lds_copies();   // no copy into LDS outlives the wavefront
        return;
    }
    const ChainHead h = walk_into_lds(t, ci, s, ls, ln, lane);   // its final wait covers the ASR row too
    constexpr int kTaken = int32_t(0x80000000u);
    float bx = -__builtin_inff();
    int bi = kNone;
    for (int c = 0; c < V; c += kStripe) {   // lane l: tokens c + 4l .. c + 4l + 3, rewritten in place
        const int v0 = c + 4 * lane;
        f32x4 x = *reinterpret_cast<const f32x4 *>(ls + v0);
        i32x4 n = *reinterpret_cast<const i32x4 *>(ln + v0);
        const f32x4 a = *reinterpret_cast<const f32x4 *>(arow + v0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float lm;
            int nx;
            slot_value(h, x[j], n[j], lm, nx);
            x[j] = __builtin_fmaf(lambda, lm, a[j]);
            n[j] = v0 + j < V ? nx : kTaken;   // padding past V counts as taken
            if (v0 + j < V) take_max(x[j], v0 + j, bx, bi);
        }
        *reinterpret_cast<f32x4 *>(ls + v0) = x;
        *reinterpret_cast<i32x4 *>(ln + v0) = n;
    }
    for (int j = 0; j < k; ++j) {
        float wv;
        int w = wave_argmax(bx, bi, wv);
        if (w == kNone) {   // everything left is -inf: the lowest index not yet taken
            int lo = kNone;
            for (int c = 0; c < V && lo == kNone; c += kStripe) {
                const int v0 = c + 4 * lane;
                const i32x4 n = *reinterpret_cast<const i32x4 *>(ln + v0);
#pragma unroll
                for (int q = 3; q >= 0; --q)
                    if (n[q] >= 0) lo = v0 + q;
            }
            w = int(~wave_max_u32(~(unsigned)lo));
        }
        if (lane == ((w & (kStripe - 1)) >> 2)) {   // the lane that owns token w
            otok[j] = w;
            osc[j] = ls[w];
            onx[j] = ln[w];
            ln[w] = ln[w] | kTaken;
            bx = -__builtin_inff();
            bi = kNone;
            for (int c = 0; c < V; c += kStripe) {
                const int v0 = c + 4 * lane;
                const f32x4 x = *reinterpret_cast<const f32x4 *>(ls + v0);
                const i32x4 n = *reinterpret_cast<const i32x4 *>(ln + v0);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (n[q] >= 0) take_max(x[q], v0 + q, bx, bi);
            }
        }
    }
}

// Inclusive prefix sum over the lanes of a wave (the DPP pattern of
// wave_max_u32 with additions).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ unsigned add_step(unsigned x) {
    return x + unsigned(__builtin_amdgcn_update_dpp(0, int(x), CTRL, ROW_MASK, 0xf, true));
}

__device__ __forceinline__ unsigned wave_incl_sum(unsigned x) {
    x = add_step<0x111, 0xf>(x);
    x = add_step<0x112, 0xf>(x);
    x = add_step<0x114, 0xf>(x);
    x = add_step<0x118, 0xf>(x);
    x = add_step<0x142, 0xa>(x);
    x = add_step<0x143, 0xc>(x);
    return x;
}

__device__ __forceinline__ unsigned wave_sum(unsigned x) {
    return unsigned(__builtin_amdgcn_readlane(int(wave_incl_sum(x)), kWave - 1));
}

// The k (distinct) sort keys in sk[0, k), with their scores and next states,
// written out in descending key order: lane l ranks entries l + 64 r (r < NR,
// k <= 64 NR) by counting the keys above them.
template <int NR>
__device__ __forceinline__ void rank_and_store(const unsigned long long *sk, const float *ssc, const int *snx, int k,
                                               int lane, int32_t *otok, float *osc, int32_t *onx) {
    unsigned long long mine[NR];
    int rank[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        mine[r] = lane + r * kWave < k ? sk[lane + r * kWave] : ~0ull;
        rank[r] = 0;
    }
#pragma unroll 8
    for (int q = 0; q < k; ++q) {
        const unsigned long long o = sk[q];
#pragma unroll
        for (int r = 0; r < NR; ++r) rank[r] += o > mine[r] ? 1 : 0;
    }
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int e = lane + r * kWave;
        if (e < k) {
            otok[rank[r]] = int(~unsigned(mine[r] & 0xffffffffu));
            osc[rank[r]] = ssc[e];
            onx[rank[r]] = snx[e];
        }
    }
}

// The same selection in a number of steps that does not grow with k (V <=
// 256 * SPL): keys are the order-preserving images of the fused values
// (value_key; tokens past V get 0, below every token's key).
//   1. the threshold T, the largest key with at least k keys >= T (the k-th
//      largest key), by a binary search over its bits: a count of the keys
//      >= a candidate is a compare and add per register slot and one wave sum
//      (DPP).  The bits that a lower bound of T and the largest key share are
//      T's from the start, and the search stops as soon as a candidate has
//      exactly k keys >= it: then those are the k taken and no tie is cut;
//   2. every key above T is taken, and of the keys equal to T the lowest
//      token indices until k are taken (a token's rank among them from
//      ballots and lane-prefix counts: token 256 c + 4 l + j sits in slot
//      4 c + j of lane l, so index order is (c, lane, j));
//   3. the k taken entries are compacted into LDS as 64-bit sort keys
//      (value key, ~index) with their score and next state, and each lands
//      at its rank, the number of taken keys above it (keys are distinct).
template <int SPL>
__global__ __launch_bounds__(kWave) void fused_topk_select_kernel(DevTrie t, const float *__restrict__ asr,
                                                                  int64_t B, int64_t ld, float lambda, int k,
                                                                  const int32_t *__restrict__ states,
                                                                  int32_t *__restrict__ tokens,
                                                                  float *__restrict__ scores,
                                                                  int32_t *__restrict__ next) {
    constexpr int kN = 4 * SPL;
    extern __shared__ float lds[];
    load_trie_args(t);
    load_args(asr, B, ld, lambda, k, states, tokens, scores, next);
    const int lane = threadIdx.x;
    const int64_t b = blockIdx.x;
    if (b >= B) return;
    const int V = t.vocab_size;
    float *ls = lds;
    int *ln = reinterpret_cast<int *>(ls + lds_row(V));
    float *arow = reinterpret_cast<float *>(ln + lds_row(V));
    int32_t *otok = tokens + b * k;
    float *osc = scores + b * k;
    int32_t *onx = next + b * k;
    const int s_l = states[b];   // issued before the row copy, so its wait leaves the copy in flight
    copy_to_lds_dword(asr + b * ld, arow, V, lane);
    const ChainIndex ci = chain_index(t, lane);
    const int s = __builtin_amdgcn_readfirstlane(s_l);
    if (s < 0 || s >= t.num_states) {
        if (lane == 0) atomicAdd(&t.status[0], 1);
        for (int j = lane; j < k; j += kWave) {
            otok[j] = -1;
            osc[j] = NAN;
            onx[j] = -1;
        }
        wait_lds_copies();   // no copy into LDS outlives the wavefront
        return;
    }
    const ChainHead h = walk_into_lds(t, ci, s, ls, ln, lane);   // its final wait covers the ASR row too
    // slot i = 4 c + j of this lane is token 256 c + 4 lane + j
    float f[kN];
    int n[kN];
    unsigned key[kN];
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
        const int v0 = c * kStripe + 4 * lane;
        const f32x4 x = *reinterpret_cast<const f32x4 *>(ls + v0);
        const i32x4 m = *reinterpret_cast<const i32x4 *>(ln + v0);
        const f32x4 a = *reinterpret_cast<const f32x4 *>(arow + v0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float lm;
            slot_value(h, x[j], m[j], lm, n[4 * c + j]);
            f[4 * c + j] = __builtin_fmaf(lambda, lm, a[j]);
            key[4 * c + j] = v0 + j < V ? value_key(f[4 * c + j]) : 0u;
        }
    }
    // 1. the threshold T.  It lies between a lower bound lo (for k <= 64 j,
    // the smallest over the lanes of a lane's j-th largest key: at least
    // 64 j >= k keys are >= it; 0 for k > 128) and the largest key, so the
    // bits above the highest one in which those two differ are T's already.
    unsigned lo = 0, mx = 0;
    if (k <= 2 * kWave) {
        unsigned m1 = 0, m2 = 0;   // the lane's largest and second largest key
#pragma unroll
        for (int i = 0; i < kN; ++i) {
            m2 = max(m2, min(m1, key[i]));
            m1 = max(m1, key[i]);
        }
        mx = wave_max_u32(m1);
        lo = ~wave_max_u32(~(k <= kWave ? m1 : m2));
    } else {
        unsigned m1 = 0;
#pragma unroll
        for (int i = 0; i < kN; ++i) m1 = max(m1, key[i]);
        mx = wave_max_u32(m1);
    }
    const unsigned diff = lo ^ mx;
    const int top = diff ? 31 - __builtin_clz(diff) : -1;
    unsigned T = top < 0 ? mx : mx & ~((2u << top) - 1u);   // top = 31: no bit known (2u << 31 is 0)
    bool exact = false;   // the keys >= T number exactly k
    for (int bit = top; bit >= 0 && !exact; --bit) {
        const unsigned cand = T | (1u << bit);
        unsigned c = 0;
#pragma unroll
        for (int i = 0; i < kN; ++i) c += key[i] >= cand ? 1u : 0u;
        const int cnt = int(wave_sum(c));
        if (cnt >= k) T = cand;
        exact = cnt == k;
    }
    int above = k;
    if (!exact) {   // T is the k-th key itself: count the keys above it
        unsigned c = 0;
#pragma unroll
        for (int i = 0; i < kN; ++i) c += key[i] > T ? 1u : 0u;
        above = int(wave_sum(c));
    }
    // 2. taken entries: every key >= T when exact; otherwise T is the k-th
    // key itself, `above` keys exceed it, and of the keys equal to it the
    // lowest token indices are taken (bit i of tie_taken: slot i is such a tie)
    unsigned tie_taken = 0;
    if (!exact) {
        const int ties_needed = k - above;
        int ties_before = 0;   // ties at T in earlier stripes (uniform)
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            unsigned long long m[4];
            int below = 0;      // ties of this stripe in lower lanes
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                m[j] = __ballot(key[4 * c + j] == T);
                below += int(__builtin_amdgcn_mbcnt_hi(unsigned(m[j] >> 32),
                                                       __builtin_amdgcn_mbcnt_lo(unsigned(m[j]), 0u)));
            }
            int own = 0;        // ties of this lane in earlier slots of the stripe
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int i = 4 * c + j;
                const bool tie = key[i] == T;
                if (tie && ties_before + below + own < ties_needed) tie_taken |= 1u << i;
                own += tie ? 1 : 0;
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) ties_before += __builtin_popcountll(m[j]);
        }
    }
    // 3. compaction into LDS (the walked row is in registers now), then ranks;
    // the exact case tests its keys directly, with no per-slot flags to build
    unsigned long long *sk = reinterpret_cast<unsigned long long *>(lds);
    float *ssc = reinterpret_cast<float *>(sk + k);
    int *snx = reinterpret_cast<int *>(ssc + k);
    auto compact = [&](auto taken) {
        int base = 0;
#pragma unroll
        for (int i = 0; i < kN; ++i) {
            const bool tk = taken(i);
            const unsigned long long m = __ballot(tk);
            if (tk) {
                const int p = base + int(__builtin_amdgcn_mbcnt_hi(unsigned(m >> 32),
                                                                  __builtin_amdgcn_mbcnt_lo(unsigned(m), 0u)));
                const int tok = (i >> 2) * kStripe + 4 * lane + (i & 3);
                sk[p] = (static_cast<unsigned long long>(key[i]) << 32) | unsigned(~unsigned(tok));
                ssc[p] = f[i];
                snx[p] = n[i];
            }
            base += __builtin_popcountll(m);
        }
    };
    if (exact)
        compact([&](int i) { return key[i] >= T; });
    else
        compact([&](int i) { return key[i] > T || ((tie_taken >> i) & 1u) != 0; });
    if (k <= kWave)
        rank_and_store<1>(sk, ssc, snx, k, lane, otok, osc, onx);
    else if (k <= 2 * kWave)
        rank_and_store<2>(sk, ssc, snx, k, lane, otok, osc, onx);
    else
        rank_and_store<4>(sk, ssc, snx, k, lane, otok, osc, onx);
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
    const size_t lds = (2 * size_t(lds_row(t.vocab_size)) + size_t(asr_row_words(t.vocab_size))) * sizeof(float);
    const dim3 grid(static_cast<unsigned>(B)), block(kWave);
    const int spl = (t.vocab_size + kStripe - 1) / kStripe;   // stripes per lane
    // V <= 1024: the selection with the row in registers, for every k (from
    // k = 6 on it beats one reduction per selected token; below that the two
    // are level: 10.1-10.5 us either way at k = 1 to 5 for 1024 hypotheses of
    // the 20M 6-gram).  Larger V: one reduction per selected token.  The k
    // taken entries (16 bytes each) may need more LDS than the row.
    const size_t lds_sel = lds > 16 * size_t(k) ? lds : 16 * size_t(k);
    switch (spl) {
        case 1:
            hipLaunchKernelGGL(fused_topk_select_kernel<1>, grid, block, lds_sel, stream, t, asr, B, ld, lambda, k,
                               states, tokens, scores, next);
            break;
        case 2:
            hipLaunchKernelGGL(fused_topk_select_kernel<2>, grid, block, lds_sel, stream, t, asr, B, ld, lambda, k,
                               states, tokens, scores, next);
            break;
        case 3:
            hipLaunchKernelGGL(fused_topk_select_kernel<3>, grid, block, lds_sel, stream, t, asr, B, ld, lambda, k,
                               states, tokens, scores, next);
            break;
        case 4:
            hipLaunchKernelGGL(fused_topk_select_kernel<4>, grid, block, lds_sel, stream, t, asr, B, ld, lambda, k,
                               states, tokens, scores, next);
            break;
        default:
            hipLaunchKernelGGL(fused_topk_kernel, grid, block, lds, stream, t, asr, B, ld, lambda, k, states, tokens,
                               scores, next);
    }
    return hipGetLastError();
}

// Wavefronts per hypothesis: a batch of up to 512 hypotheses leaves most SIMDs
// idle with one wavefront each, so each hypothesis gets four (measured on the
// 20M 6-gram decode: 4-12 % less time per frame); from 1024 on, one wavefront
// per hypothesis keeps more work in flight and wins.
inline int waves_per_hyp(int64_t B) { return B <= 512 ? 4 : 1; }

// The same choice for one step per launch, where every launch pays the whole
// dependent chain once: four wavefronts stay ahead up to 1024 hypotheses
// (20M 6-gram, CTC: 8.54 against 8.70 us per step at 768, 8.95 against 9.12
// at 1024; 11.2 against 10.6 at 2048).
inline int step_waves_per_hyp(int64_t B) { return B <= 1024 ? 4 : 1; }

// Wavefronts that own one 256-token stripe each load only their stripe's part
// of every sparse level.
template <int W>
inline bool stripe_split(const DevTrie &t) {
    return W > 1 && (t.vocab_size + kStripe - 1) / kStripe == W;
}

template <int MODE, int W>
static hipError_t launch_step_w(const DevTrie &t, const float *asr, int64_t B, int64_t ld, float lambda,
                                int32_t *states, int32_t *prev, int32_t *tokens, hipStream_t stream) {
    if constexpr (W > 1) {
        if (stripe_split<W>(t)) {
            hipLaunchKernelGGL((fused_step_kernel<MODE, W, true>), dim3(unsigned(B)), dim3(W * kWave),
                               hyp_lds_bytes(t.vocab_size, 1), stream, t, asr, B, ld, lambda, states, prev, tokens);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((fused_step_kernel<MODE, W, false>), dim3(unsigned(B)), dim3(W * kWave),
                       hyp_lds_bytes(t.vocab_size, 1), stream, t, asr, B, ld, lambda, states, prev, tokens);
    return hipGetLastError();
}

template <int MODE>
static hipError_t launch_step_mode(const DevTrie &t, const float *asr, int64_t B, int64_t ld, float lambda,
                                   int32_t *states, int32_t *prev, int32_t *tokens, hipStream_t stream) {
    switch (step_waves_per_hyp(B)) {
        case 4: return launch_step_w<MODE, 4>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        default: return launch_step_w<MODE, 1>(t, asr, B, ld, lambda, states, prev, tokens, stream);
    }
}

hipError_t launch_fused_step(const DevTrie &t, const float *asr, int64_t B, int64_t ld, int mode, float lambda,
                             int32_t *states, int32_t *prev, int32_t *tokens, hipStream_t stream) {
    switch (mode) {
        case kPlain: return launch_step_mode<kPlain>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        case kCtc: return launch_step_mode<kCtc>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        case kAed: return launch_step_mode<kAed>(t, asr, B, ld, lambda, states, prev, tokens, stream);
        default: return launch_step_mode<kTransducer>(t, asr, B, ld, lambda, states, prev, tokens, stream);
    }
}

template <int MODE, int W, int NB, bool FULL = false>
static hipError_t launch_decode_w(const DevTrie &t, const float *asr, int64_t B, int64_t T, int64_t sb, int64_t st,
                                  const int32_t *lengths, float lambda, int32_t *states, int32_t *prev,
                                  int32_t *labels, int32_t *label_states, hipStream_t stream) {
    if constexpr (W > 1) {
        if (stripe_split<W>(t)) {
            hipLaunchKernelGGL((fused_decode_kernel<MODE, W, NB, FULL, true>), dim3(unsigned(B)), dim3(W * kWave),
                               hyp_lds_bytes(t.vocab_size, NB), stream, t, asr, B, T, sb, st, lengths, lambda, states,
                               prev, labels, label_states);
            return hipGetLastError();
        }
    }
    if constexpr (W == 1 && NB == 0) {
        if (t.dense_c) {
            hipLaunchKernelGGL((fused_decode_kernel<MODE, 1, 0, FULL, false, true>), dim3(unsigned(B)), dim3(kWave),
                               hyp_lds_bytes(t.vocab_size, 0), stream, t, asr, B, T, sb, st, lengths, lambda, states,
                               prev, labels, label_states);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((fused_decode_kernel<MODE, W, NB, FULL, false>), dim3(unsigned(B)), dim3(W * kWave),
                       hyp_lds_bytes(t.vocab_size, NB), stream, t, asr, B, T, sb, st, lengths, lambda, states, prev,
                       labels, label_states);
    return hipGetLastError();
}

// Utterances the device holds at once with two ASR row buffers per utterance
// (one wavefront each): CUs times the workgroups whose LDS fits one CU.  The
// two device attributes are queried once per device and kept (a decode call
// then costs one hipGetDevice on the host for this).
static int64_t resident_double_buffered(const DevTrie &t) {
    constexpr int kMaxDevices = 64;
    static std::atomic<int64_t> cached[kMaxDevices];   // CUs << 32 | LDS bytes per CU; 0: not yet known
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
        (void)hipGetLastError();
        return INT64_MAX;   // unknown: keep two buffers
    }
    int64_t c = dev < kMaxDevices ? cached[dev].load(std::memory_order_relaxed) : 0;
    if (c == 0) {
        int cus = 0, lds = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) != hipSuccess ||
            cus <= 0 || lds <= 0) {
            (void)hipGetLastError();
            return INT64_MAX;
        }
        c = (int64_t(cus) << 32) | int64_t(uint32_t(lds));
        if (dev < kMaxDevices) cached[dev].store(c, std::memory_order_relaxed);
    }
    const int64_t cus = c >> 32, lds = c & 0xffffffff;
    return cus * int64_t(size_t(lds) / hyp_lds_bytes(t.vocab_size, 2));
}

template <int MODE>
static hipError_t launch_decode_mode(const DevTrie &t, const float *asr, int64_t B, int64_t T, int64_t sb,
                                     int64_t st, const int32_t *lengths, float lambda, int32_t *states,
                                     int32_t *prev, int32_t *labels, int32_t *label_states, hipStream_t stream) {
    if (waves_per_hyp(B) == 4)
        return launch_decode_w<MODE, 4, 2>(t, asr, B, T, sb, st, lengths, lambda, states, prev, labels, label_states,
                                           stream);
    // Measured on the 20M 6-gram, CTC, 200 frames: with compact dense rows
    // the register rows are the fastest at every size (0.556 / 0.571 / 0.611
    // / 0.625 / 0.654 ms against 0.624 / 0.638 / 0.696 / 0.705 / 0.789 ms for
    // two LDS row buffers at 600 / 1024 / 1536 / 2048 / 2304 utterances).
    // Without them: while every utterance is resident with two LDS row
    // buffers (2304 utterances on 256 CUs at V = 1024), those are 2-4 % faster
    // than rows in registers; beyond that the register rows (up to 16
    // utterances per CU) are 27 % faster at 4096 utterances and 18 % at 8192,
    // and one LDS buffer (13 per CU) still beats two by 8-14 %.
    if (!(t.dense_c && t.vocab_size <= kRegTokens) && B <= resident_double_buffered(t))
        return launch_decode_w<MODE, 1, 2>(t, asr, B, T, sb, st, lengths, lambda, states, prev, labels, label_states,
                                           stream);
    if (t.vocab_size == kRegTokens)
        return launch_decode_w<MODE, 1, 0, true>(t, asr, B, T, sb, st, lengths, lambda, states, prev, labels,
                                                 label_states, stream);
    if (t.vocab_size < kRegTokens)
        return launch_decode_w<MODE, 1, 0>(t, asr, B, T, sb, st, lengths, lambda, states, prev, labels, label_states,
                                           stream);
    return launch_decode_w<MODE, 1, 1>(t, asr, B, T, sb, st, lengths, lambda, states, prev, labels, label_states,
                                       stream);
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
