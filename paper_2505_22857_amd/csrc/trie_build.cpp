// Host construction of the trie image from a closed n-gram list (Section 2.2);
// with NGPU_BUILD_REPAIR_CLOSURE a list that is not closed is closed first.
//
// Every n-gram is packed into a 128-bit key, ceil(log2 V) bits per token with
// the first token most significant, so that numeric order of keys of one order
// is lexicographic order of the tuples.  Per order the keys are sorted; a
// state's id is then 1 + (number of shorter contexts) + its rank, which equals
// the canonical numbering (order, tuple).  The prefix of an order-k key is
// key >> bits and its suffix is the low (k-1)*bits bits, so the closure checks,
// the backoff state (the suffix) and the arc ranges (children share the prefix)
// are binary searches and scans over the sorted keys.  The image then holds,
// per state, its whole backoff chain (arc ranges and accumulators), dense rows
// for the empty context and the order-1 states, and the sparse arcs of the
// deeper states (layout in trie.h).
#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>

#include "trie.h"

namespace ngpu {
namespace {

typedef unsigned __int128 u128;

struct Entry {
    u128 key;
    int64_t row;
};

struct OrderLevel {
    std::vector<u128> key;        // sorted
    std::vector<float> w, b;      // weight / backoff in sorted order
    std::vector<int32_t> prefix;  // rank of the prefix in order k-1 (k >= 2)
    std::vector<int32_t> suffix;  // rank of the suffix in order k-1 (k >= 2)
};

int bits_for(int32_t V) {
    int b = 1;
    while ((int64_t(1) << b) < V) ++b;
    return b;
}

// rank of key in sorted keys, or -1
int64_t find_rank(const std::vector<u128> &keys, u128 k) {
    auto it = std::lower_bound(keys.begin(), keys.end(), k);
    if (it == keys.end() || *it != k) return -1;
    return it - keys.begin();
}

std::string tuple_text(u128 key, int k, int bits) {
    std::string s = "(";
    for (int i = 0; i < k; ++i) {
        uint64_t t = uint64_t(key >> (bits * (k - 1 - i))) & ((uint64_t(1) << bits) - 1);
        if (i) s += ' ';
        s += std::to_string(t);
    }
    return s + ")";
}

// Closure repair (NGPU_BUILD_REPAIR_CLOSURE): every missing prefix and suffix
// of a listed n-gram (for n-grams ending in </s>, the prefix only) is inserted
// with backoff 0 and the weight the backoff rule gives it on the list without
// it.  Missing n-grams are collected from the highest order down (an inserted
// n-gram needs its own prefix and suffix), then weighted from order 1 up:
// for an inserted x = c + v of order k >= 2 the rule stops at the suffix x[1:],
// which is present, so W(x) = B(c) + W(x[1:]) (one fp32 add, B(c) = 0 when c
// was inserted too); an inserted unigram takes the <unk> weight.  Scores of
// every history are unchanged (the rule adds B = 0 for an unlisted context),
// and the inserted contexts become states the walk can reach.
int repair_closure(std::vector<OrderLevel> &lv, int N, int bits, bool has_unk, float unk,
                   const std::vector<std::pair<u128, int>> &final_ctx, std::string *err, int64_t *inserted) {
    std::vector<std::vector<char>> ins(N + 1);
    for (int k = 1; k <= N; ++k) ins[k].assign(lv[k].key.size(), 0);
    *inserted = 0;
    for (int k = N; k >= 1; --k) {
        // missing (k-1)-grams: prefixes and suffixes of order-k n-grams, prefixes (contexts) of finals of order k
        std::vector<u128> need;
        if (k >= 2) {
            const u128 smask = (u128(1) << (bits * (k - 1))) - 1;
            for (const u128 &x : lv[k].key) {
                need.push_back(x >> bits);
                need.push_back(x & smask);
            }
        }
        for (const auto &f : final_ctx)
            if (f.second == k - 1 && k >= 2) need.push_back(f.first);
        if (k == 1) break;
        std::sort(need.begin(), need.end());
        need.erase(std::unique(need.begin(), need.end()), need.end());
        OrderLevel &L = lv[k - 1];
        std::vector<u128> add;
        for (const u128 &x : need)
            if (!std::binary_search(L.key.begin(), L.key.end(), x)) add.push_back(x);
        if (add.empty()) continue;
        // merge the additions into the sorted level, weights filled in below
        const size_t n0 = L.key.size(), n1 = n0 + add.size();
        std::vector<u128> key(n1);
        std::vector<float> w(n1), b(n1);
        std::vector<char> mark(n1);
        size_t i = 0, j = 0;
        for (size_t p = 0; p < n1; ++p) {
            if (j >= add.size() || (i < n0 && L.key[i] < add[j])) {
                key[p] = L.key[i];
                w[p] = L.w[i];
                b[p] = L.b[i];
                mark[p] = ins[k - 1][i];
                ++i;
            } else {
                key[p] = add[j];
                w[p] = 0.0f;
                b[p] = 0.0f;
                mark[p] = 1;
                ++j;
            }
        }
        L.key.swap(key);
        L.w.swap(w);
        L.b.swap(b);
        ins[k - 1].swap(mark);
        *inserted += int64_t(add.size());
    }
    for (int k = 1; k <= N; ++k) {
        OrderLevel &L = lv[k];
        const u128 smask = (u128(1) << (bits * (k - 1))) - 1;
        for (size_t p = 0; p < L.key.size(); ++p) {
            if (!ins[k][p]) continue;
            if (k == 1) {
                if (!has_unk) {
                    *err = "repair needs the unigram " + tuple_text(L.key[p], 1, bits) + " but no <unk> weight was given";
                    return NGPU_E_MISSING_UNIGRAM;
                }
                L.w[p] = unk;
                continue;
            }
            const int64_t pr = find_rank(lv[k - 1].key, L.key[p] >> bits);
            const int64_t sr = find_rank(lv[k - 1].key, L.key[p] & smask);
            L.w[p] = lv[k - 1].b[size_t(pr)] + lv[k - 1].w[size_t(sr)];
        }
    }
    return NGPU_OK;
}

}  // namespace

int build_trie(const ngpu_ngram_list *list, int32_t V, float unk, uint32_t flags, ngpu_lm *lm, std::string *err) {
    const int N = list->max_order;
    const int64_t M = list->num_ngrams;
    // with <s> and </s>: token V is <s> (only first), V + 1 is </s> (only last)
    const bool special = (flags & NGPU_BUILD_BOS_EOS) != 0;
    const int32_t bos = V, eos = V + 1;
    const int32_t Vt = special ? V + 2 : V;
    if (N < 1 || N > NGPU_LM_MAX_ORDER) {
        *err = "max_order must be in [1, " + std::to_string(NGPU_LM_MAX_ORDER) + "]";
        return NGPU_E_ORDER_RANGE;
    }
    if (V < 1 || V > NGPU_LM_MAX_VOCAB) {
        *err = "vocab_size must be in [1, " + std::to_string(NGPU_LM_MAX_VOCAB) + "]";
        return NGPU_E_TOO_LARGE;
    }
    const int bits = bits_for(Vt);
    if (bits * N > 128) {
        *err = "ceil(log2 V) * max_order exceeds 128 bits";
        return NGPU_E_TOO_LARGE;
    }
    if (M < 0 || (M > 0 && (!list->order || !list->tokens || !list->logprob || !list->backoff))) {
        *err = "null n-gram arrays";
        return NGPU_E_INVALID_ARG;
    }
    if (M > int64_t(INT32_MAX) - 1) {
        *err = "too many n-grams for int32 state and arc ids";
        return NGPU_E_TOO_LARGE;
    }
    const bool has_unk = !std::isnan(unk);
    if (has_unk && !std::isfinite(unk)) {
        *err = "unk_logprob must be finite or NaN";
        return NGPU_E_NONFINITE;
    }

    // ---- bucket by order, validate, pack keys
    std::vector<int64_t> count(N + 1, 0);
    for (int64_t i = 0; i < M; ++i) {
        int k = list->order[i];
        if (k < 1 || k > N) {
            *err = "row " + std::to_string(i) + ": order " + std::to_string(k) + " outside [1, max_order]";
            return NGPU_E_ORDER_RANGE;
        }
        ++count[k];
    }
    std::vector<std::vector<Entry>> ent(N + 1);
    for (int k = 1; k <= N; ++k) ent[k].reserve(count[k]);
    struct Final {
        u128 ctx;
        int order;   // context order
        int64_t row;
    };
    std::vector<Final> finals;   // n-grams ending in </s>: final weights of their contexts
    for (int64_t i = 0; i < M; ++i) {
        int k = list->order[i];
        const int32_t *t = list->tokens + i * N;
        u128 key = 0;
        for (int j = 0; j < k; ++j) {
            if (t[j] < 0 || t[j] >= Vt) {
                *err = "row " + std::to_string(i) + ": token " + std::to_string(t[j]) + " outside [0, " +
                       std::to_string(Vt) + ")";
                return NGPU_E_TOKEN_RANGE;
            }
            if (special && ((t[j] == bos && j != 0) || (t[j] == eos && j != k - 1))) {
                *err = "row " + std::to_string(i) + ": <s> may only open and </s> only close an n-gram";
                return NGPU_E_TOKEN_RANGE;
            }
            key = (key << bits) | u128(uint32_t(t[j]));
        }
        const bool ends_eos = special && t[k - 1] == eos;
        if (!std::isfinite(list->logprob[i]) || (k < N && !ends_eos && !std::isfinite(list->backoff[i]))) {
            *err = "row " + std::to_string(i) + ": non-finite weight";
            return NGPU_E_NONFINITE;
        }
        if (ends_eos) finals.push_back({key >> bits, k - 1, i});
        else ent[k].push_back({key, i});
    }

    std::vector<OrderLevel> lv(N + 1);
    for (int k = 1; k <= N; ++k) {
        auto &e = ent[k];
        std::sort(e.begin(), e.end(), [](const Entry &a, const Entry &b) { return a.key < b.key; });
        OrderLevel &L = lv[k];
        L.key.resize(e.size());
        L.w.resize(e.size());
        L.b.resize(e.size());
        for (size_t p = 0; p < e.size(); ++p) {
            if (p && e[p].key == e[p - 1].key) {
                *err = "duplicate n-gram " + tuple_text(e[p].key, k, bits);
                return NGPU_E_DUPLICATE_NGRAM;
            }
            L.key[p] = e[p].key;
            L.w[p] = list->logprob[e[p].row];
            L.b[p] = k < N ? list->backoff[e[p].row] : 0.0f;
        }
        std::vector<Entry>().swap(e);
    }
    if (flags & NGPU_BUILD_REPAIR_CLOSURE) {
        std::vector<std::pair<u128, int>> final_ctx;
        for (const Final &f : finals)
            if (f.order > 0) final_ctx.push_back({f.ctx, f.order});
        int64_t added = 0;
        const int rc = repair_closure(lv, N, bits, has_unk, unk, final_ctx, err, &added);
        if (rc != NGPU_OK) return rc;
    }
    {
        int64_t regular = 0;   // unigrams of scored tokens (not <s>)
        for (const u128 &k1 : lv[1].key) regular += k1 < u128(uint32_t(V)) ? 1 : 0;
        if (!has_unk && regular < V) {
            *err = "a token has no unigram and no <unk> weight was given";
            return NGPU_E_MISSING_UNIGRAM;
        }
        if (special && find_rank(lv[1].key, u128(uint32_t(bos))) < 0) {
            *err = "<s> has no unigram, so there is no start state";
            return NGPU_E_MISSING_UNIGRAM;
        }
    }

    // ---- closure: prefix and suffix of every order-k n-gram are listed
    for (int k = 2; k <= N; ++k) {
        OrderLevel &L = lv[k];
        const std::vector<u128> &low = lv[k - 1].key;
        const u128 smask = (u128(1) << (bits * (k - 1))) - 1;
        const size_t n = L.key.size();
        L.prefix.resize(n);
        L.suffix.resize(n);
        for (size_t p = 0; p < n; ++p) {
            int64_t pr = find_rank(low, L.key[p] >> bits);
            if (pr < 0) {
                *err = "n-gram " + tuple_text(L.key[p], k, bits) + " has no listed prefix";
                return NGPU_E_MISSING_PREFIX;
            }
            int64_t sr = find_rank(low, L.key[p] & smask);
            if (sr < 0) {
                *err = "n-gram " + tuple_text(L.key[p], k, bits) + " has no listed suffix";
                return NGPU_E_MISSING_SUFFIX;
            }
            L.prefix[p] = int32_t(pr);
            L.suffix[p] = int32_t(sr);
        }
    }

    // ---- ids: state (k, rank) -> first[k] + rank for k < N; arcs: order k >= 2 at arc_base[k] + rank
    std::vector<int64_t> first(N + 1, 0), arc_base(N + 2, 0);
    int64_t S = 1;
    for (int k = 1; k < N; ++k) {
        first[k] = S;
        S += int64_t(lv[k].key.size());
    }
    int64_t A = 0;
    for (int k = 2; k <= N; ++k) {
        arc_base[k] = A;
        A += int64_t(lv[k].key.size());
    }
    if (S > INT32_MAX || A > INT32_MAX) {
        *err = "too many states or arcs for int32 ids";
        return NGPU_E_TOO_LARGE;
    }
    if (S > NGPU_LM_MAX_STATES) {
        *err = std::to_string(S) + " states exceed the " + std::to_string(NGPU_LM_MAX_STATES) +
               " that 30-bit state ids hold";
        return NGPU_E_TOO_LARGE;
    }

    // ---- host CSR records over the host arc numbering (orders 2..N at arc_base[k])
    std::vector<StateRec> rec(static_cast<size_t>(S));
    rec[0] = StateRec{0, 0, 0.0f, 0};
    lm->state_parent.assign(size_t(S), 0);
    lm->state_tok.assign(size_t(S), -1);
    const uint64_t tmask = (uint64_t(1) << bits) - 1;
    for (int k = 1; k < N; ++k) {
        const OrderLevel &L = lv[k];
        const size_t n = L.key.size();
        // children of (k, p) are the order-(k+1) n-grams whose prefix rank is p, contiguous
        const std::vector<int32_t> &cp = lv[k + 1].prefix;
        size_t c = 0;
        for (size_t p = 0; p < n; ++p) {
            size_t c0 = c;
            while (c < cp.size() && cp[c] == int32_t(p)) ++c;
            int64_t id = first[k] + int64_t(p);
            rec[id].begin = int32_t(arc_base[k + 1] + int64_t(c0));
            rec[id].end = int32_t(arc_base[k + 1] + int64_t(c));
            rec[id].bw = L.b[p];
            rec[id].bto = k == 1 ? 0 : int32_t(first[k - 1] + L.suffix[p]);
            lm->state_parent[id] = k == 1 ? 0 : int32_t(first[k - 1] + L.prefix[p]);
            lm->state_tok[id] = int32_t(uint64_t(L.key[p]) & tmask);
        }
    }
    const int64_t n1 = N > 1 ? int64_t(lv[1].key.size()) : 0;   // order-1 states
    const int64_t A3 = N >= 3 ? A - int64_t(lv[2].key.size()) : 0;  // arcs of orders >= 3
    const int64_t arc3 = N >= 3 ? arc_base[3] : 0;                  // host index of the first one
    const int64_t R = 1 + n1;                                       // dense rows

    // ---- image layout
    ImageHeader h{};
    h.magic = kImageMagic;
    h.vocab_size = V;
    h.max_order = N;
    h.dense_rows = int32_t(R);
    h.num_states = S;
    h.num_arcs = A3;
    for (int k = 0; k <= NGPU_LM_MAX_ORDER; ++k) h.first[k] = int32_t(k == 0 ? 0 : (k < N ? first[k] : S));
    size_t off = align_up(sizeof(ImageHeader));
    h.off_status = off;
    off = align_up(off + 4 * sizeof(int32_t));
    h.off_chain = off;
    size_t coff = 0;
    for (int k = 0; k < N; ++k) {
        h.off_order[k] = coff;
        const int64_t cnt = k == 0 ? 1 : (k + 1 < N ? first[k + 1] : S) - first[k];
        coff += size_t(cnt) * 16 * size_t(k == 0 ? 1 : k);
    }
    off = align_up(off + coff);
    h.off_dense_w = off;
    off = align_up(off + size_t(R) * size_t(V) * 4);
    h.off_dense_to = off;
    off = align_up(off + size_t(R) * size_t(V) * 4);
    // arcs of order N: the only ones whose next state is not their own n-gram's
    const int64_t top_begin = N >= 3 ? arc_base[N] - arc3 : 0;
    h.top_arc_begin = top_begin;
    h.arc_to_delta = N > 3 ? int32_t(first[3]) : 0;
    h.off_arcs = off;
    off = align_up(off + size_t(top_begin) * sizeof(Arc));
    h.off_top_arcs = off;
    off = align_up(off + size_t(A3 - top_begin) * sizeof(TopArc));
    h.has_final = special ? 1 : 0;
    h.off_final = special ? off : 0;
    if (special) off = align_up(off + size_t(S) * 4);
    // compact dense rows (for the whole decode with rows in registers): room
    // is made when the vocabulary allows them, and given back below if the
    // model does not qualify
    const size_t off_without_compact = off;
    const bool try_compact = V >= 2 && V <= 1024 && N >= 2;
    h.compact_rank = N > 2 ? 1 : 0;
    if (try_compact) {
        h.off_dense_c = off;
        off = align_up(off + size_t(R) * size_t(V) * 4);
        h.off_dense_base = off;
        off = align_up(off + size_t(R) * 4);
    }
    h.start_state = 0;
    if (special && N > 1) h.start_state = int32_t(first[1] + find_rank(lv[1].key, u128(uint32_t(bos))));
    h.total_bytes = off;

    std::vector<unsigned char> img;
    try {
        img.assign(off, 0);
    } catch (const std::bad_alloc &) {
        *err = "host allocation of the trie image failed";
        return NGPU_E_NO_MEMORY;
    }
    std::memcpy(img.data(), &h, sizeof h);
    unsigned char *chain = img.data() + h.off_chain;
    float *dense_w = reinterpret_cast<float *>(img.data() + h.off_dense_w);
    int32_t *dense_to = reinterpret_cast<int32_t *>(img.data() + h.off_dense_to);
    Arc *arcs = reinterpret_cast<Arc *>(img.data() + h.off_arcs);
    TopArc *top_arcs = reinterpret_cast<TopArc *>(img.data() + h.off_top_arcs);
    // token of image arc a (either array)
    auto arc_tok = [&](int64_t a) { return a < top_begin ? arcs[a].tok : top_arcs[a - top_begin].tok; };

    // dense row 0: the empty context (Section 2.2: every token has an arc; missing ones get <unk>)
    for (int32_t v = 0; v < V; ++v) {
        dense_w[v] = has_unk ? unk : 0.0f;
        dense_to[v] = 0;
    }
    for (size_t p = 0; p < lv[1].key.size(); ++p) {
        int32_t v = int32_t(uint64_t(lv[1].key[p]));
        if (v >= V) continue;   // <s> is a context only, never scored
        dense_w[v] = lv[1].w[p];
        dense_to[v] = N > 1 ? int32_t(first[1] + int64_t(p)) : 0;
    }
    // dense rows of the order-1 states: own bigrams, else the empty-context entry flagged
    for (int64_t u = 1; u <= n1; ++u) {
        float *rw = dense_w + size_t(u) * size_t(V);
        int32_t *rt = dense_to + size_t(u) * size_t(V);
        for (int32_t v = 0; v < V; ++v) {
            rw[v] = dense_w[v];
            rt[v] = dense_to[v] | kDenseBackoff;
        }
        const OrderLevel &L2 = lv[2];
        for (int32_t a = rec[u].begin; a < rec[u].end; ++a) {   // order-2 arcs: host index = rank
            int32_t v = int32_t(uint64_t(L2.key[a]) & tmask);
            rw[v] = L2.w[a];
            rt[v] = N > 2 ? int32_t(first[2] + a) : int32_t(first[1] + L2.suffix[a]);
        }
    }
    // compact dense rows: the weight's magnitude with the sign bit as the
    // backoff flag; kept only if every weight's sign bit is set and the
    // next-state rules reproduce dense_to for every entry
    if (try_compact) {
        float *dc = reinterpret_cast<float *>(img.data() + h.off_dense_c);
        int32_t *db = reinterpret_cast<int32_t *>(img.data() + h.off_dense_base);
        bool ok = true;
        for (int64_t u = 0; u < R && ok; ++u) {
            const float *rw = dense_w + size_t(u) * size_t(V);
            const int32_t *rt = dense_to + size_t(u) * size_t(V);
            float *rc = dc + size_t(u) * size_t(V);
            int32_t base = u == 0 ? int32_t(first[1]) : -1, rank = 0;
            for (int32_t v = 0; v < V && ok; ++v) {
                uint32_t wb;
                std::memcpy(&wb, &rw[v], 4);
                const bool backoff = (rt[v] & kDenseBackoff) != 0;
                const int32_t to = rt[v] & ~kDenseBackoff;
                const uint32_t cb = backoff ? wb : (wb & 0x7fffffffu);
                std::memcpy(&rc[v], &cb, 4);
                int64_t want = first[1] + v;
                if (!backoff && h.compact_rank) {   // own entry (every entry of row 0)
                    if (base < 0) base = to;
                    want = int64_t(base) + rank++;
                }
                ok = (wb & 0x80000000u) && to == want;
            }
            db[u] = base < 0 ? 0 : base;
        }
        if (!ok) {
            h.off_dense_c = 0;
            h.off_dense_base = 0;
            off = off_without_compact;
            h.total_bytes = off;
            img.resize(off);
            std::memcpy(img.data(), &h, sizeof h);
        }
    }

    // sparse arcs of orders 3..N: token and weight; the next state is the
    // arc's own n-gram (k < N: first[k] + p = a + first[3], as arc_base[k] -
    // arc3 and first[k] - first[3] both count the orders 3 .. k-1) or, for
    // order N, the n-gram's suffix
    for (int k = 3; k <= N; ++k) {
        const OrderLevel &L = lv[k];
        for (size_t p = 0; p < L.key.size(); ++p) {
            int64_t a = arc_base[k] - arc3 + int64_t(p);
            const int32_t tok = int32_t(uint64_t(L.key[p]) & tmask);
            if (k < N) {
                arcs[a].tok = tok;
                arcs[a].w = L.w[p];
            } else {
                TopArc &ta = top_arcs[a - top_begin];
                ta.tok = tok;
                ta.w = L.w[p];
                ta.to = int32_t(first[N - 1] + L.suffix[p]);
            }
        }
    }
    // dense-row groups: longest-processing-time assignment of rows, weighted by
    // the number of states whose chain ends in the row, to kGroups bins
    std::vector<int64_t> row_weight(size_t(R), 0);
    row_weight[0] = 1;
    for (int k = 1; k < N; ++k) {
        const int64_t end = k + 1 < N ? first[k + 1] : S;
        for (int64_t s0 = first[k]; s0 < end; ++s0) {
            int64_t s = s0;
            for (int j = 0; j < k - 1; ++j) s = rec[s].bto;
            ++row_weight[size_t(s)];
        }
    }
    std::vector<int32_t> row_group(size_t(R), 0);
    {
        std::vector<int64_t> order(static_cast<size_t>(R));
        std::iota(order.begin(), order.end(), int64_t(0));
        std::stable_sort(order.begin(), order.end(),
                         [&](int64_t a, int64_t b) { return row_weight[a] > row_weight[b]; });
        int64_t load[kGroups] = {0};
        for (int64_t r : order) {
            int g = 0;
            for (int i = 1; i < kGroups; ++i)
                if (load[i] < load[g]) g = i;
            row_group[size_t(r)] = g;
            load[g] += row_weight[size_t(r)];
        }
    }

    // token-stripe splits of each state's arcs (V <= 1024 only): the number of
    // arcs with token below 256, 512 and 768, packed as 9 + 10 + 10 bits, so
    // that a query split over the 256-token stripes finds its part of a level
    // without searching (arcs are sorted by token)
    std::vector<uint32_t> splits;
    if (V <= 4 * 256) {
        splits.assign(size_t(S), 0u);
        for (int64_t st = first[2 < N ? 2 : N]; N >= 3 && st < S; ++st) {
            uint32_t c[3] = {0, 0, 0};
            for (int32_t a = rec[st].begin; a < rec[st].end; ++a) {
                const int32_t tok = arc_tok(a - arc3);
                for (int i = 0; i < 3; ++i) c[i] += tok < 256 * (i + 1) ? 1u : 0u;
            }
            splits[size_t(st)] = c[0] | (c[1] << 9) | (c[2] << 19);
        }
    }

    // chain records: the fp32 fold of backoff weights from the state downward
    {
        ChainHead root{0, 0.0f, 0.0f, row_group[0] << 16};   // the empty context: dense row 0, no sparse level
        std::memcpy(chain, &root, sizeof root);
    }
    for (int k = 1; k < N; ++k) {
        const int64_t end = k + 1 < N ? first[k + 1] : S;
        for (int64_t s0 = first[k]; s0 < end; ++s0) {
            unsigned char *r = chain + h.off_order[k] + size_t(s0 - first[k]) * 16 * size_t(k);
            ChainLevel *lev = reinterpret_cast<ChainLevel *>(r + 16);
            float acc = 0.0f;
            int64_t s = s0;
            for (int j = 0; j < k - 1; ++j) {   // states of order k, k-1, ..., 2
                lev[j].begin = int32_t(rec[s].begin - arc3);
                lev[j].end = int32_t(rec[s].end - arc3);
                lev[j].acc = acc;
                lev[j].splits = splits.empty() ? 0u : splits[size_t(s)];
                acc = acc + rec[s].bw;
                s = rec[s].bto;
            }
            ChainHead hd;
            hd.dense_row = int32_t(s);           // the order-1 ancestor: state id u is dense row u
            hd.acc1 = acc;
            hd.acc0 = acc + rec[s].bw;
            hd.nlev_group = (k - 1) | (row_group[size_t(s)] << 16);
            std::memcpy(r, &hd, sizeof hd);
        }
    }

    // final weights: the </s> score of every state, by the same fp32 fold as a
    // query (the first state on the chain that lists </s> adds its weight)
    if (special) {
        std::vector<float> expl(size_t(S), 0.0f);
        std::vector<char> has(size_t(S), 0);
        std::sort(finals.begin(), finals.end(), [](const Final &a, const Final &b) {
            return a.order != b.order ? a.order < b.order : a.ctx < b.ctx;
        });
        for (size_t i = 0; i < finals.size(); ++i) {
            const Final &f = finals[i];
            if (i && f.order == finals[i - 1].order && f.ctx == finals[i - 1].ctx) {
                *err = "duplicate </s> n-gram";
                return NGPU_E_DUPLICATE_NGRAM;
            }
            int64_t st = 0;
            if (f.order > 0) {
                const int64_t r = find_rank(lv[f.order].key, f.ctx);
                if (r < 0) {
                    *err = "an n-gram ending in </s> has no listed context";
                    return NGPU_E_MISSING_PREFIX;
                }
                st = first[f.order] + r;
            }
            expl[size_t(st)] = list->logprob[f.row];
            has[size_t(st)] = 1;
        }
        if (!has[0] && !has_unk) {
            *err = "</s> has no unigram and no <unk> weight was given";
            return NGPU_E_MISSING_UNIGRAM;
        }
        float *fin = reinterpret_cast<float *>(img.data() + h.off_final);
        for (int64_t s0 = 0; s0 < S; ++s0) {
            float acc = 0.0f;
            int64_t x = s0;
            for (int lvl = 0; lvl <= N; ++lvl) {
                if (has[size_t(x)]) {
                    fin[s0] = acc + expl[size_t(x)];
                    break;
                }
                if (x == 0) {
                    fin[s0] = acc + unk;
                    break;
                }
                acc = acc + rec[size_t(x)].bw;
                x = rec[size_t(x)].bto;
            }
        }
    }

    lm->V = V;
    lm->N = N;
    lm->S = S;
    lm->A = A;
    lm->hdr = h;
    lm->rec.swap(rec);
    lm->image.swap(img);
    return NGPU_OK;
}

}  // namespace ngpu
