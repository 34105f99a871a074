// Batched full-vocabulary backoff query (Algorithm 1, batched over hypotheses).
//
// One wavefront per hypothesis, HPB wavefronts per workgroup, each with its
// own V-wide score/state row in LDS (8 bytes per token).  After the walk
// (dense row copied in, sparse levels applied on top), the row is written to
// HBM with 16-byte non-temporal stores (when V is a multiple of 4): lane l
// covers tokens 4l..4l+3 of each 256-token stripe, so one store instruction
// of the wavefront writes 1 KiB contiguously.
//
// XCD-aware distribution (G = 8): workgroups are dispatched round-robin over
// the eight XCDs, so workgroup i serves dense-row group i % 8.  Each wavefront
// scans G consecutive hypotheses (lane i loads the state and chain head of
// hypothesis i, two vector loads) and processes the ones whose dense row lies
// in its group; the eight workgroups of a chunk together cover every
// hypothesis exactly once.  Each XCD's L2 then holds an eighth of the dense
// rows instead of all of them.  G = 1 is the plain one-hypothesis-per-wave
// mapping.  Small batches (latency-bound) give each hypothesis one wavefront
// per 256-token stripe instead (advance_striped_kernel).  No MFMA: the work is
// gathers, scatters and one fp32 add per token.
#include <hip/hip_runtime.h>

#include <cmath>

#include "walk.h"

namespace ngpu {

typedef float nf4 __attribute__((ext_vector_type(4)));
typedef int ni4 __attribute__((ext_vector_type(4)));

template <int HPB, bool VEC, int G>
__global__ __launch_bounds__(HPB * kWave) void advance_kernel(DevTrie t, const int32_t *__restrict__ states,
                                                               int64_t B, float *__restrict__ scores,
                                                               int32_t *__restrict__ next) {
    extern __shared__ float lds[];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int grp = int(blockIdx.x % G);
    const int64_t base = (int64_t(blockIdx.x / G) * HPB + wave) * G;
    if (base >= B) return;  // whole wavefronts leave; no workgroup barrier is used
    const int V = t.vocab_size;
    float *ls = lds + size_t(wave) * 2 * lds_row(V);
    int *ln = reinterpret_cast<int *>(ls + lds_row(V));

    // scan: lane i < G looks at hypothesis base + i
    int s_l = -1, dense_l = -1;
    bool mine = false;
    const int64_t bl = base + lane;
    if (lane < G && bl < B) {
        s_l = states[bl];
        if (s_l < 0 || s_l >= t.num_states) {
            s_l = -1;
            mine = (bl % G) == grp;   // an invalid state's row is written by one owner
        } else if (G == 1) {
            mine = true;
        } else {
            int nl;
            const ChainHead hd = *reinterpret_cast<const ChainHead *>(chain_record(t, s_l, nl));
            mine = chain_group(hd) == grp;
            dense_l = hd.dense_row;   // lets the walk start the dense-row copy before the record load
        }
    }
    // The scan's loads are complete here; otherwise the wait for them stays at
    // the head of the loop below, where it would also drain the previous
    // hypothesis's stores before the next one's loads are issued.
    wait_loads();
    uint64_t todo = __ballot(mine);
    const KernargTables ci;
    while (todo) {
        const int i = __builtin_ctzll(todo);
        todo &= todo - 1;
        const int64_t b = base + i;
        float *orow = scores + b * V;
        int32_t *nrow = next + b * V;
        const int s = __builtin_amdgcn_readlane(s_l, i);
        if (s < 0) {
            if (lane == 0) atomicAdd(&t.status[0], 1);
            for (int v = lane; v < V; v += kWave) {
                orow[v] = NAN;
                nrow[v] = -1;
            }
            continue;
        }
        const ChainHead h = G == 1 ? walk_into_lds(t, ci, s, ls, ln, lane)
                                   : walk_into_lds_dense_first(t, ci, s, __builtin_amdgcn_readlane(dense_l, i), ls,
                                                               ln, lane);
        if (VEC) {
            for (int v = lane * 4; v < V; v += 4 * kWave) {
                const int4 n4 = *reinterpret_cast<const int4 *>(ln + v);
                const float4 x4 = *reinterpret_cast<const float4 *>(ls + v);
                nf4 xo;
                ni4 no;
                float x;
                int n;
                slot_value(h, x4.x, n4.x, x, n); xo.x = x; no.x = n;
                slot_value(h, x4.y, n4.y, x, n); xo.y = x; no.y = n;
                slot_value(h, x4.z, n4.z, x, n); xo.z = x; no.z = n;
                slot_value(h, x4.w, n4.w, x, n); xo.w = x; no.w = n;
                // streaming stores: the rows are not read again here, so they
                // should not displace the dense rows and arcs from the L2
                __builtin_nontemporal_store(xo, reinterpret_cast<nf4 *>(orow + v));
                __builtin_nontemporal_store(no, reinterpret_cast<ni4 *>(nrow + v));
            }
        } else {
            for (int v = lane; v < V; v += kWave) {
                float x;
                int n;
                slot_value(h, ls[v], ln[v], x, n);
                __builtin_nontemporal_store(x, orow + v);
                __builtin_nontemporal_store(n, nrow + v);
            }
        }
    }
}

// The XCD-grouped mapping with two wavefronts per hypothesis, independent of
// each other: part p walks and writes tokens [512 p, 512 p + 512) through its
// own 4 KiB LDS row, loading only its half of every level (the split counts:
// arcs are sorted by token).  Half the LDS per wavefront lets more of them,
// and their stores, be in flight per CU.  V in (768, 1024], a multiple of 4.
template <int G>
__global__ __launch_bounds__(kWave) void advance_half_kernel(DevTrie t, const int32_t *__restrict__ states, int64_t B,
                                                             float *__restrict__ scores,
                                                             int32_t *__restrict__ next) {
    extern __shared__ float lds[];
    const int lane = threadIdx.x;
    const int grp = int(blockIdx.x % G);
    const int part = int((blockIdx.x / G) & 1);
    const int64_t base = int64_t(blockIdx.x / (2 * G)) * G;
    if (base >= B) return;
    const int V = t.vocab_size;
    const int c0 = 2 * kStripe * part;   // slot of token v: v - c0
    float *ls = lds;
    int *ln = reinterpret_cast<int *>(lds + 2 * kStripe);

    int s_l = -1, dense_l = -1;
    bool mine = false;
    const int64_t bl = base + lane;
    if (lane < G && bl < B) {
        s_l = states[bl];
        if (s_l < 0 || s_l >= t.num_states) {
            s_l = -1;
            mine = (bl % G) == grp;
        } else {
            int nl;
            const ChainHead hd = *reinterpret_cast<const ChainHead *>(chain_record(t, s_l, nl));
            mine = chain_group(hd) == grp;
            dense_l = hd.dense_row;
        }
    }
    wait_loads();   // as in advance_kernel
    uint64_t todo = __ballot(mine);
    const KernargTables ci;
    while (todo) {
        const int i = __builtin_ctzll(todo);
        todo &= todo - 1;
        const int64_t b = base + i;
        float *orow = scores + b * V;
        int32_t *nrow = next + b * V;
        const int s = __builtin_amdgcn_readlane(s_l, i);
        if (s < 0) {
            if (lane == 0 && part == 0) atomicAdd(&t.status[0], 1);
            for (int v = c0 + lane; v < V && v < c0 + 2 * kStripe; v += kWave) {
                orow[v] = NAN;
                nrow[v] = -1;
            }
            continue;
        }
        dense_half_to_lds(t, __builtin_amdgcn_readlane(dense_l, i), ls, ln, part, lane);
        int nlev;
        const int4 rec = fetch_record(t, ci, s, lane, nlev);
        const ChainHead h = walk_record<1, false, true, true>(t, rec, nlev, ls, ln, lane, part);
        for (int c = c0; c < V && c < c0 + 2 * kStripe; c += kStripe) {
            const int v = c + 4 * lane;
            if (v < V) {
                const int4 n4 = *reinterpret_cast<const int4 *>(ln + (v - c0));
                const float4 x4 = *reinterpret_cast<const float4 *>(ls + (v - c0));
                nf4 xo;
                ni4 no;
                float x;
                int n;
                slot_value(h, x4.x, n4.x, x, n); xo.x = x; no.x = n;
                slot_value(h, x4.y, n4.y, x, n); xo.y = x; no.y = n;
                slot_value(h, x4.z, n4.z, x, n); xo.z = x; no.z = n;
                slot_value(h, x4.w, n4.w, x, n); xo.w = x; no.w = n;
                __builtin_nontemporal_store(xo, reinterpret_cast<nf4 *>(orow + v));
                __builtin_nontemporal_store(no, reinterpret_cast<ni4 *>(nrow + v));
            }
        }
    }
}

// The same query with W wavefronts per hypothesis: wavefront w owns the
// 256-token stripes c with c mod W = w, copies their dense entries, applies
// the sparse arcs that fall in them and writes them out, so the wavefronts
// never wait for each other (no barrier) and each writes a W-th of the row.
template <int W, bool VEC, bool SPLIT>
__global__ __launch_bounds__(W * kWave) void advance_striped_kernel(DevTrie t, const int32_t *__restrict__ states,
                                                                     int64_t B, float *__restrict__ scores,
                                                                     int32_t *__restrict__ next) {
    extern __shared__ float lds[];
    load_trie_args(t);
    load_args(states, B, scores, next);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int64_t b = blockIdx.x;
    if (b >= B) return;
    const int V = t.vocab_size;
    float *ls = lds;
    int *ln = reinterpret_cast<int *>(ls + lds_row(V));
    float *orow = scores + b * V;
    int32_t *nrow = next + b * V;
    const int s = __builtin_amdgcn_readfirstlane(states[b]);
    const ChainIndex ci = chain_index(t, lane);
    if (s < 0 || s >= t.num_states) {
        if (wave == 0 && lane == 0) atomicAdd(&t.status[0], 1);
        for (int v = wave * kWave + lane; v < V; v += W * kWave) {
            orow[v] = NAN;
            nrow[v] = -1;
        }
        return;
    }
    int nlev;
    const int4 rec = fetch_record(t, ci, s, lane, nlev);
    const ChainHead h = walk_record<W, SPLIT>(t, rec, nlev, ls, ln, lane, wave);
    for (int c = kStripe * wave; c < V; c += kStripe * W) {
        if (VEC) {
            const int v = c + 4 * lane;
            if (v < V) {   // V is a multiple of 4, so v + 3 < V too
                const int4 n4 = *reinterpret_cast<const int4 *>(ln + v);
                const float4 x4 = *reinterpret_cast<const float4 *>(ls + v);
                nf4 xo;
                ni4 no;
                float x;
                int n;
                slot_value(h, x4.x, n4.x, x, n); xo.x = x; no.x = n;
                slot_value(h, x4.y, n4.y, x, n); xo.y = x; no.y = n;
                slot_value(h, x4.z, n4.z, x, n); xo.z = x; no.z = n;
                slot_value(h, x4.w, n4.w, x, n); xo.w = x; no.w = n;
                __builtin_nontemporal_store(xo, reinterpret_cast<nf4 *>(orow + v));
                __builtin_nontemporal_store(no, reinterpret_cast<ni4 *>(nrow + v));
            }
        } else {
            for (int v = c + lane; v < V && v < c + kStripe; v += kWave) {
                float x;
                int n;
                slot_value(h, ls[v], ln[v], x, n);
                __builtin_nontemporal_store(x, orow + v);
                __builtin_nontemporal_store(n, nrow + v);
            }
        }
    }
}

// SPLIT when the wavefronts own one stripe each (V in (256 (W - 1), 256 W]):
// each then loads only its stripe's part of every level.
template <int W>
static hipError_t launch_striped(const DevTrie &t, const int32_t *states, int64_t B, float *scores, int32_t *next,
                                 hipStream_t stream, bool vec) {
    const size_t lds = 2 * size_t(lds_row(t.vocab_size)) * sizeof(float);
    const bool split = W > 1 && (t.vocab_size + kStripe - 1) / kStripe == W;
    const dim3 grid(static_cast<unsigned>(B)), block(W * kWave);
    if (vec && split)
        hipLaunchKernelGGL((advance_striped_kernel<W, true, true>), grid, block, lds, stream, t, states, B, scores,
                           next);
    else if (vec)
        hipLaunchKernelGGL((advance_striped_kernel<W, true, false>), grid, block, lds, stream, t, states, B, scores,
                           next);
    else if (split)
        hipLaunchKernelGGL((advance_striped_kernel<W, false, true>), grid, block, lds, stream, t, states, B, scores,
                           next);
    else
        hipLaunchKernelGGL((advance_striped_kernel<W, false, false>), grid, block, lds, stream, t, states, B, scores,
                           next);
    return hipGetLastError();
}

template <int HPB, int G>
static hipError_t launch_hpb(const DevTrie &t, const int32_t *states, int64_t B, float *scores,
                             int32_t *next, hipStream_t stream, bool vec) {
    const int64_t chunks = (B + int64_t(HPB) * G - 1) / (int64_t(HPB) * G);
    const dim3 grid(unsigned(chunks * G)), block(HPB * kWave);
    const size_t lds = size_t(HPB) * 2 * size_t(lds_row(t.vocab_size)) * sizeof(float);
    if (vec)
        hipLaunchKernelGGL((advance_kernel<HPB, true, G>), grid, block, lds, stream, t, states, B, scores, next);
    else
        hipLaunchKernelGGL((advance_kernel<HPB, false, G>), grid, block, lds, stream, t, states, B, scores, next);
    return hipGetLastError();
}

// Launch shapes, from a sweep on the 20M n-gram workload (V = 1024):
//  - XCD-grouped mapping from 20480 hypotheses on; below that the grouped
//    scan costs more latency than the cache locality saves (grouped against
//    plain: 48.3 / 46.9 us at 18000, 49.4 / 52.2 at 20480, 62.4 / 70.1 at
//    28672, 67.5 / 79.3 at 32767).
//  - One wavefront per workgroup in the grouped mapping: a wavefront that finds
//    no hypothesis of its group frees its slot (and LDS) at once instead of
//    waiting for busier wavefronts of its workgroup.
//  - Two wavefronts per workgroup in the plain mapping.
//  - Up to 1024 hypotheses, where a call is latency-bound, four wavefronts per
//    hypothesis, each walking and writing its own stripes: 8.6 against
//    9.4 us at 128 hypotheses, 9.0 against 9.9 at 512, 9.6 against 10.0 at
//    1024; 10.7 against 10.5 at 1536 and 12.1 against 11.2 at 2048.
constexpr int64_t kStripedMaxBatch = 1024;
constexpr int64_t kGroupedMinBatch = 20480;
constexpr int kHpbGrouped = 1;
constexpr int kHpbPlain = 2;

// Wavefronts per workgroup: at most `want`, as many rows as fit in 32 KiB of LDS.
int rows_per_block(int V, int want) {
    const size_t row = size_t(lds_row(V)) * 8;
    int h = want;
    while (h > 1 && size_t(h) * row > 32768) h /= 2;
    return h;
}

hipError_t launch_advance(const DevTrie &t, const int32_t *states, int64_t B, float *scores, int32_t *next,
                          hipStream_t stream) {
    const bool vec = (t.vocab_size % 4 == 0) && (reinterpret_cast<uintptr_t>(scores) % 16 == 0) &&
                     (reinterpret_cast<uintptr_t>(next) % 16 == 0);
    if (B >= kGroupedMinBatch) {
        const int64_t chunks = (B + kGroups - 1) / kGroups;
        if (vec && (t.vocab_size + kStripe - 1) / kStripe == 4 &&
            2 * chunks * kGroups * kWave <= int64_t(UINT32_MAX)) {   // dispatch size in work-items
            hipLaunchKernelGGL(advance_half_kernel<kGroups>, dim3(unsigned(2 * chunks * kGroups)), dim3(kWave),
                               size_t(4 * kStripe) * sizeof(float), stream, t, states, B, scores, next);
            return hipGetLastError();
        }
        return launch_hpb<kHpbGrouped, kGroups>(t, states, B, scores, next, stream, vec);
    }
    if (B <= kStripedMaxBatch) {   // wavefronts per hypothesis: one per stripe, at most four
        const int stripes = (t.vocab_size + kStripe - 1) / kStripe;
        if (stripes >= 4) return launch_striped<4>(t, states, B, scores, next, stream, vec);
        if (stripes >= 2) return launch_striped<2>(t, states, B, scores, next, stream, vec);
        return launch_striped<1>(t, states, B, scores, next, stream, vec);
    }
    switch (rows_per_block(t.vocab_size, kHpbPlain)) {
        case 2: return launch_hpb<2, 1>(t, states, B, scores, next, stream, vec);
        default: return launch_hpb<1, 1>(t, states, B, scores, next, stream, vec);
    }
}

}  // namespace ngpu
