// Internal layout of the trie image shared by the host builder, the C ABI and
// the HIP kernels of this library.
//
// The image is one contiguous byte buffer, identical on host and device, with
// 256-byte aligned sections (offsets in ImageHeader):
//   status   int32 [4]   device-written counters ([0]: out-of-range input states)
//   chain    per state, its whole backoff chain, grouped by order k and
//            addressed as chain + off_order[k] + (s - first[k]) * 16 * max(k, 1):
//              ChainHead {dense_row, acc1, acc0, nlev | group << 16}
//              ChainLevel[nlev] {arc_begin, arc_end, acc, splits}   (orders k, k-1, ..., 2)
//            The accumulators are the fp32 left fold of the backoff weights
//            from the query state downward (Algorithm 1), computed on the host
//            in the same order the walk would take, so they are bit-identical
//            to a walk that adds them one by one.
//   dense_w  float [R * V]  dense rows: row 0 is the empty context (unigram or
//   dense_to int32 [R * V]  <unk> weight), row u = 1..n1 is the order-1 state u:
//            its own bigram weight and state where listed, else the
//            empty-context entry with DENSE_BACKOFF set in dense_to (that
//            token's score takes acc0 instead of acc1).  Each dense row belongs
//            to one of kGroups groups, balanced by the number of states whose
//            chain ends in it; a query kernel may serve each group from one XCD
//            so that the group's rows stay in that XCD's L2.
//   arcs     arcs of states of order >= 2 (n-grams of order >= 3), sorted by
//            (from_state, token) (Section 2.2), numbered 0 .. A3 - 1; 64 lanes
//            read 64 arcs of a level with one load instruction.  An arc of
//            order k < N leads to the state of its own n-gram, and states and
//            arcs of one order share their sorted order, so its next state is
//            its index plus arc_to_delta (= first[3]):
//              Arc {token, weight} [top_arc_begin]           orders 3 .. N-1
//            The arcs of order N lead to their n-gram's suffix and keep it:
//   top_arcs TopArc {token, weight, next} [A3 - top_arc_begin]   order N
//   final    float [S]   with </s> in the model: each state's end-of-sentence
//                        weight, folded through its backoff chain at build
//                        time (Section 2.3, AED)
//   dense_c    float [R * V]  the dense rows again in 4 bytes per token, for
//   dense_base int32 [R]      the whole-decode kernel that holds rows in
//            registers, which needs a token's next state only for the frame's
//            winner: dense_c is the weight's magnitude, its sign bit set where
//            the entry backed off to the empty context (DENSE_BACKOFF), so
//            weight = dense_c with the sign bit set.  A backed-off token v (and
//            every token of row 0) leads to the unigram state first[1] + v; an
//            own bigram of row u leads to dense_base[u] + the number of own
//            bigrams of row u below it when compact_rank is set (orders >= 3:
//            bigrams are states, numbered in the row's token order), else to
//            first[1] + v.  Present (off_dense_c != 0) only when V <= 1024,
//            every dense weight has its sign bit set and these rules give
//            dense_to exactly for every entry, which the builder checks.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "ngpu_lm.h"

namespace ngpu {

constexpr uint32_t kImageMagic = 0x354d4c4e;  // "NLM5"
constexpr size_t kAlign = 256;
constexpr int32_t kDenseBackoff = int32_t(0x80000000u);  // flag bit in dense_to
constexpr int kGroups = 8;                                // dense-row groups (one per XCD)

struct ImageHeader {
    uint32_t magic;
    int32_t vocab_size;
    int32_t max_order;
    int32_t dense_rows;
    int64_t num_states;
    int64_t num_arcs;            // sparse arcs in the image (orders >= 3)
    uint64_t off_status, off_chain, off_dense_w, off_dense_to, off_arcs;
    uint64_t total_bytes;
    int32_t first[NGPU_LM_MAX_ORDER + 1];       // first state id of each order; first[N] = S
    uint64_t off_order[NGPU_LM_MAX_ORDER];      // chain offset (from the chain section) per order
    uint64_t off_final;                         // final weights float[S] (0 when the model has no </s>)
    int32_t start_state;                        // state of the context <s> (0 without <s>)
    int32_t has_final;
    uint64_t off_top_arcs;                      // the order-N arcs
    int64_t top_arc_begin;                      // first arc of order N (A3 when there is none)
    int32_t arc_to_delta;                       // next state of arc a of order < N: a + arc_to_delta
    int32_t compact_rank;                       // dense_c: own bigrams numbered by their rank in the row
    uint64_t off_dense_c;                       // compact dense rows (0 when the model does not qualify)
    uint64_t off_dense_base;                    // int32[R]: first own-bigram state of each dense row
};
static_assert(sizeof(ImageHeader) == 264, "the header layout is part of the image format");

struct ChainHead {
    int32_t dense_row;
    float acc1;   // accumulator at the order-1 ancestor: applies to its own bigrams
    float acc0;   // accumulator at the empty context: applies to backed-off tokens
    int32_t nlev_group;   // number of sparse levels | dense-row group << 16
};
struct ChainLevel {
    int32_t begin;
    int32_t end;
    float acc;
    uint32_t splits;   // V <= 1024: arcs with token < 256 | < 512 << 9 | < 768 << 19; else 0
};
static_assert(sizeof(ChainHead) == 16 && sizeof(ChainLevel) == 16, "chain records are 16-byte units");

struct Arc {
    int32_t tok;
    float w;
};
static_assert(sizeof(Arc) == 8, "an arc below the highest order is two words");
struct TopArc {
    int32_t tok;
    float w;
    int32_t to;
};
static_assert(sizeof(TopArc) == 12, "an arc of the highest order is three words");

// Host-side CSR record (not in the device image): used for byte accounting.
struct StateRec {
    int32_t begin;  // into the host arc numbering (orders >= 2)
    int32_t end;
    float bw;
    int32_t bto;
};

// Kernel view of an uploaded image.
struct DevTrie {
    const unsigned char *chain;
    const float *dense_w;
    const int32_t *dense_to;
    const Arc *arcs;          // arcs 0 .. top_begin - 1
    const TopArc *top_arcs;   // arcs top_begin .. A3 - 1, at a - top_begin
    const float *final_w;   // nullptr without </s>
    int32_t *status;
    const float *dense_c;         // nullptr when the model has no compact dense rows
    const int32_t *dense_base;
    int32_t num_states;
    int32_t vocab_size;
    int32_t max_order;
    int32_t top_begin;      // first arc of the highest order
    int32_t to_delta;       // next state of an arc below top_begin: its index + to_delta
    int32_t compact_rank;
    int32_t first[NGPU_LM_MAX_ORDER + 1];
    uint64_t off_order[NGPU_LM_MAX_ORDER];
};

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

}  // namespace ngpu

struct ngpu_lm {
    int32_t V = 0, N = 0;
    int64_t S = 0, A = 0;                 // A: arcs of orders >= 2 (host numbering)
    std::vector<unsigned char> image;     // host copy of the device image
    ngpu::ImageHeader hdr{};
    std::vector<ngpu::StateRec> rec;      // [S] CSR records over the host arc numbering
    std::vector<int32_t> state_parent;    // [S] state of the context minus its last token
    std::vector<int32_t> state_tok;       // [S] last token of the context
    void *dev = nullptr;                  // uploaded image (caller-owned)
    int device = -1;
};

namespace ngpu {
// api.cpp: records the thread's last error message and returns code
int set_error(int code, const std::string &msg);
// trie_build.cpp
int build_trie(const ngpu_ngram_list *list, int32_t V, float unk, uint32_t flags, ngpu_lm *lm, std::string *err);
}  // namespace ngpu
