// Internal layout of the trie image shared by the host builder, the C ABI and
// the HIP kernels of this library.
//
// The image is one contiguous byte buffer, identical on host and device, with
// 256-byte aligned sections (offsets in ImageHeader):
//   rec      int4  [S]  per state {arc_begin, arc_end, backoff weight bits, backoff state}
//                       (Section 2.2: start_arcs/end_arcs ranges, boff_weights,
//                       boff_to_states); state 0 (empty context) has an empty range
//   root_w   float [V]  dense row of the empty context: unigram weight, or <unk>
//   root_to  int32 [V]  next state of each unigram arc (0 for <unk> tokens)
//   arc_tok  int32 [A]  arcs of non-empty contexts, sorted by (from_state, token)
//   arc_w    float [A]
//   arc_to   int32 [A]
//   status   int32 [4]  device-written counters ([0]: out-of-range input states)
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "ngpu_lm.h"

namespace ngpu {

constexpr uint32_t kImageMagic = 0x4d4c504e;  // "NPLM"
constexpr size_t kAlign = 256;

struct ImageHeader {
    uint32_t magic;
    int32_t vocab_size;
    int32_t max_order;
    int32_t pad0;
    int64_t num_states;
    int64_t num_arcs;
    uint64_t off_rec, off_root_w, off_root_to, off_arc_tok, off_arc_w, off_arc_to, off_status;
    uint64_t total_bytes;
};

struct StateRec {
    int32_t begin;
    int32_t end;
    float bw;
    int32_t bto;
};
static_assert(sizeof(StateRec) == 16, "state record must be 16 bytes");

// Kernel view of an uploaded image.
struct DevTrie {
    const StateRec *rec;
    const float *root_w;
    const int32_t *root_to;
    const int32_t *arc_tok;
    const float *arc_w;
    const int32_t *arc_to;
    int32_t *status;
    int32_t num_states;
    int32_t vocab_size;
    int32_t max_order;
};

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

}  // namespace ngpu

struct ngpu_lm {
    int32_t V = 0, N = 0;
    int64_t S = 0, A = 0;
    std::vector<unsigned char> image;     // host copy of the device image
    ngpu::ImageHeader hdr{};
    std::vector<int64_t> state_first;     // first state id of each order 1..N-1 (index by order)
    std::vector<int32_t> state_parent;    // [S] state of the context minus its last token
    std::vector<int32_t> state_tok;       // [S] last token of the context
    void *dev = nullptr;                  // uploaded image (caller-owned)
    int device = -1;

    const ngpu::StateRec *rec() const {
        return reinterpret_cast<const ngpu::StateRec *>(image.data() + hdr.off_rec);
    }
};

namespace ngpu {
// trie_build.cpp
int build_trie(const ngpu_ngram_list *list, int32_t V, float unk, ngpu_lm *lm, std::string *err);
}  // namespace ngpu
