// ARPA text -> n-gram list (Section 2.1: one line per n-gram, "W context token B",
// weights as base-10 logarithms as KenLM writes them).
//
// Words map to ids through the caller's vocabulary (ids 0..V-1).  <unk>
// gives its unigram weight as the <unk> weight and never appears as a token:
// longer n-grams that contain it are dropped, which keeps a closed list
// closed, since every prefix or suffix of a kept n-gram is kept too.  <s> and
// </s> become ids V and V + 1 with NGPU_BUILD_BOS_EOS and are dropped the same
// way without it.  Weights are converted to natural logarithms by one
// multiplication by ln 10 in double and one rounding to fp32.
#include <algorithm>
#include <cerrno>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <string>
#include <new>
#include <unordered_map>
#include <vector>

#include "trie.h"

struct ngpu_arpa {
    int32_t max_order = 0;
    int64_t count = 0;
    std::vector<int32_t> order;
    std::vector<int32_t> tokens;   // [count * max_order], padded with -1
    std::vector<float> logprob;
    std::vector<float> backoff;
    float unk = NAN;
};

namespace {

constexpr double kLn10 = 2.302585092994045684017991454684364208;

struct Line {
    const char *p;
    const char *end;
};

bool next_line(const char *&cur, const char *end, Line &ln) {
    if (cur >= end) return false;
    const char *e = static_cast<const char *>(memchr(cur, '\n', size_t(end - cur)));
    if (!e) e = end;
    ln.p = cur;
    ln.end = e;
    while (ln.end > ln.p && (ln.end[-1] == '\r' || ln.end[-1] == ' ' || ln.end[-1] == '\t')) --ln.end;
    while (ln.p < ln.end && (*ln.p == ' ' || *ln.p == '\t')) ++ln.p;
    cur = e < end ? e + 1 : end;
    return true;
}

// Whitespace-separated fields of a line.
void split(const Line &ln, std::vector<std::string> &f) {
    f.clear();
    const char *p = ln.p;
    while (p < ln.end) {
        while (p < ln.end && (*p == ' ' || *p == '\t')) ++p;
        const char *q = p;
        while (q < ln.end && *q != ' ' && *q != '\t') ++q;
        if (q > p) f.emplace_back(p, size_t(q - p));
        p = q;
    }
}

bool parse_double(const std::string &s, double &x) {
    errno = 0;
    char *e = nullptr;
    x = std::strtod(s.c_str(), &e);
    return e && *e == '\0' && errno == 0;
}

bool starts_with(const Line &ln, const char *s) {
    const size_t n = strlen(s);
    return size_t(ln.end - ln.p) >= n && memcmp(ln.p, s, n) == 0;
}

// k of a "\k-grams:" line, else 0.
int section_of(const Line &ln) {
    const std::string s(ln.p, ln.end);
    if (s.size() < 9 || s[0] != '\\' || s.compare(s.size() - 7, 7, "-grams:") != 0) return 0;
    char *e = nullptr;
    const long k = std::strtol(s.c_str() + 1, &e, 10);
    return (e && std::string(e) == "-grams:" && k >= 1) ? int(k) : 0;
}

}  // namespace

extern "C" {

static int arpa_parse(const char *text, size_t len, const char *const *vocab, int32_t V, uint32_t flags,
                      ngpu_arpa **out);

// Host allocations inside the reader may throw; nothing may cross the C ABI.
int ngpu_arpa_parse(const char *text, size_t len, const char *const *vocab, int32_t V, uint32_t flags,
                    ngpu_arpa **out) {
    try {
        return arpa_parse(text, len, vocab, V, flags, out);
    } catch (const std::bad_alloc &) {
        if (out) *out = nullptr;   // arpa_parse frees its partial list as the exception leaves it
        return ngpu::set_error(NGPU_E_NO_MEMORY, "host allocation failed while reading the ARPA text");
    } catch (const std::exception &e) {
        if (out) *out = nullptr;
        return ngpu::set_error(NGPU_E_NO_MEMORY, std::string("ARPA reader: ") + e.what());
    }
}

static int arpa_parse(const char *text, size_t len, const char *const *vocab, int32_t V, uint32_t flags,
                      ngpu_arpa **out) {
    using ngpu::set_error;
    if (!out) return set_error(NGPU_E_INVALID_ARG, "out is null");
    *out = nullptr;
    if (!text || !vocab || V < 1 || V > NGPU_LM_MAX_VOCAB) return set_error(NGPU_E_INVALID_ARG, "bad arguments");
    if ((flags & ~NGPU_BUILD_BOS_EOS) != 0) return set_error(NGPU_E_INVALID_ARG, "unknown flags");
    const bool special = (flags & NGPU_BUILD_BOS_EOS) != 0;
    std::unordered_map<std::string, int32_t> id;
    id.reserve(size_t(V) * 2);
    for (int32_t v = 0; v < V; ++v) {
        if (!vocab[v]) return set_error(NGPU_E_INVALID_ARG, "null vocabulary entry " + std::to_string(v));
        if (!id.emplace(vocab[v], v).second)
            return set_error(NGPU_E_INVALID_ARG, std::string("duplicate vocabulary entry '") + vocab[v] + "'");
    }
    constexpr int32_t kUnk = -2, kBos = -3, kEos = -4;
    for (const char *w : {"<unk>", "<s>", "</s>"})
        if (id.count(w)) return set_error(NGPU_E_INVALID_ARG, std::string("vocabulary must not contain ") + w);
    id.emplace("<unk>", kUnk);
    id.emplace("<s>", kBos);
    id.emplace("</s>", kEos);

    std::unique_ptr<ngpu_arpa> a(new (std::nothrow) ngpu_arpa());   // freed on every early return and throw
    if (!a) return set_error(NGPU_E_NO_MEMORY, "out of host memory");
    const char *cur = text, *end = text + len;
    Line ln;
    std::vector<std::string> f;
    std::vector<int64_t> declared(NGPU_LM_MAX_ORDER + 1, -1);
    auto fail = [&](int code, const std::string &msg) { return set_error(code, msg); };
    // header
    bool in_data = false;
    int section = 0;
    while (next_line(cur, end, ln)) {
        if (ln.p == ln.end) continue;
        if (starts_with(ln, "\\data\\")) {
            in_data = true;
            continue;
        }
        if (!in_data) continue;
        if (starts_with(ln, "ngram ")) {
            std::string s(ln.p + 6, size_t(ln.end - ln.p - 6));
            const size_t eq = s.find('=');
            if (eq == std::string::npos) return fail(NGPU_E_INVALID_ARG, "bad ngram count line");
            const int k = std::atoi(s.substr(0, eq).c_str());
            if (k < 1 || k > NGPU_LM_MAX_ORDER) return fail(NGPU_E_ORDER_RANGE, "ngram order out of range");
            declared[k] = std::atoll(s.substr(eq + 1).c_str());
            a->max_order = std::max(a->max_order, k);
            continue;
        }
        if (section_of(ln)) {
            section = section_of(ln);
            break;
        }
        return fail(NGPU_E_INVALID_ARG, "unexpected line in the \\data\\ header");
    }
    if (!in_data || a->max_order < 1 || section != 1) return fail(NGPU_E_INVALID_ARG, "no \\data\\ header or 1-grams");
    const int N = a->max_order;
    std::vector<int64_t> seen(N + 1, 0);
    std::vector<int32_t> row(N);
    bool ended = false;
    while (next_line(cur, end, ln)) {
        if (ln.p == ln.end) continue;
        if (ln.p[0] == '\\') {
            if (starts_with(ln, "\\end\\")) {
                ended = true;
                break;
            }
            const int k = section_of(ln);
            if (k != section + 1 || k > N) return fail(NGPU_E_INVALID_ARG, "sections out of order");
            section = k;
            continue;
        }
        const int k = section;
        split(ln, f);
        if (int(f.size()) != k + 1 && int(f.size()) != k + 2)
            return fail(NGPU_E_INVALID_ARG, "a " + std::to_string(k) + "-gram line has " +
                                                std::to_string(f.size()) + " fields");
        ++seen[k];
        double w, b = 0.0;
        if (!parse_double(f[0], w) || (int(f.size()) == k + 2 && !parse_double(f[k + 1], b)))
            return fail(NGPU_E_NONFINITE, "unreadable weight in '" + std::string(ln.p, ln.end) + "'");
        bool keep = true, is_unk_unigram = false;
        for (int j = 0; j < k; ++j) {
            auto it = id.find(f[1 + j]);
            if (it == id.end()) return fail(NGPU_E_TOKEN_RANGE, "word '" + f[1 + j] + "' is not in the vocabulary");
            int32_t t = it->second;
            if (t == kUnk) {
                if (k == 1) is_unk_unigram = true;
                keep = false;
            } else if (t == kBos || t == kEos) {
                if (!special) keep = false;
                t = t == kBos ? V : V + 1;
            }
            row[j] = t;
        }
        if (is_unk_unigram) a->unk = float(w * kLn10);
        if (!keep) continue;
        a->order.push_back(k);
        for (int j = 0; j < N; ++j) a->tokens.push_back(j < k ? row[j] : -1);
        a->logprob.push_back(float(w * kLn10));
        a->backoff.push_back(float(b * kLn10));
    }
    if (!ended) return fail(NGPU_E_INVALID_ARG, "no \\end\\ line");
    for (int k = 1; k <= N; ++k)
        if (declared[k] >= 0 && declared[k] != seen[k])
            return fail(NGPU_E_INVALID_ARG, "the header declares " + std::to_string(declared[k]) + " " +
                                                std::to_string(k) + "-grams, the file lists " +
                                                std::to_string(seen[k]));
    a->count = int64_t(a->order.size());
    *out = a.release();
    return set_error(NGPU_OK, "");
}

int ngpu_arpa_list(const ngpu_arpa *a, ngpu_ngram_list *list, float *unk_logprob) {
    if (!a || !list || !unk_logprob) return ngpu::set_error(NGPU_E_INVALID_ARG, "null argument");
    list->num_ngrams = a->count;
    list->max_order = a->max_order;
    list->order = a->order.data();
    list->tokens = a->tokens.data();
    list->logprob = a->logprob.data();
    list->backoff = a->backoff.data();
    *unk_logprob = a->unk;
    return ngpu::set_error(NGPU_OK, "");
}

void ngpu_arpa_free(ngpu_arpa *a) { delete a; }

}  // extern "C"
