// Host-only driver of the trie builder and the ARPA reader, for builds with
// the address and undefined-behaviour sanitizers (tests/test_host_sanitizers.py).
//
//   build_driver list LIST OUT            binary n-gram list -> build
//   build_driver arpa TEXT VOCAB FLAGS OUT  ARPA text + vocabulary file (one
//                                          word per line) -> parse -> build
//
// LIST: int32 V, int32 N, int64 M, float unk, uint32 flags, then int32
// order[M], int32 tokens[M * N], float logprob[M], float backoff[M].
// Prints "rc <code>"; on success writes the built image to OUT.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <fstream>
#include <iterator>
#include <string>
#include <vector>

#include "trie.h"

namespace ngpu {
// The library's version records a thread-local message; the code is all a driver needs.
int set_error(int code, const std::string &) { return code; }
}  // namespace ngpu

namespace {

std::vector<char> slurp(const char *path) {
    std::ifstream f(path, std::ios::binary);
    return std::vector<char>((std::istreambuf_iterator<char>(f)), std::istreambuf_iterator<char>());
}

template <class T>
bool take(const std::vector<char> &buf, size_t &pos, T *dst, size_t n) {
    if (pos + n * sizeof(T) > buf.size()) return false;
    std::memcpy(dst, buf.data() + pos, n * sizeof(T));
    pos += n * sizeof(T);
    return true;
}

int finish(int rc, const ngpu_lm &lm, const char *out) {
    std::printf("rc %d\n", rc);
    if (rc == NGPU_OK) {
        std::ofstream f(out, std::ios::binary);
        f.write(reinterpret_cast<const char *>(lm.image.data()), std::streamsize(lm.image.size()));
    }
    return 0;
}

}  // namespace

int main(int argc, char **argv) {
    std::string err;
    if (argc == 4 && std::strcmp(argv[1], "list") == 0) {
        const std::vector<char> buf = slurp(argv[2]);
        size_t pos = 0;
        int32_t V = 0, N = 0;
        int64_t M = 0;
        float unk = 0;
        uint32_t flags = 0;
        if (!take(buf, pos, &V, 1) || !take(buf, pos, &N, 1) || !take(buf, pos, &M, 1) || !take(buf, pos, &unk, 1) ||
            !take(buf, pos, &flags, 1) || M < 0 || N < 1 || N > 64) {
            std::fprintf(stderr, "bad list header\n");
            return 2;
        }
        std::vector<int32_t> order(static_cast<size_t>(M)), tokens(static_cast<size_t>(M) * static_cast<size_t>(N));
        std::vector<float> W(static_cast<size_t>(M)), B(static_cast<size_t>(M));
        if (!take(buf, pos, order.data(), order.size()) || !take(buf, pos, tokens.data(), tokens.size()) ||
            !take(buf, pos, W.data(), W.size()) || !take(buf, pos, B.data(), B.size())) {
            std::fprintf(stderr, "short list file\n");
            return 2;
        }
        ngpu_ngram_list list;
        list.num_ngrams = M;
        list.max_order = N;
        list.order = order.data();
        list.tokens = tokens.data();
        list.logprob = W.data();
        list.backoff = B.data();
        ngpu_lm lm;
        const int rc = ngpu::build_trie(&list, V, unk, flags, &lm, &err);
        return finish(rc, lm, argv[3]);
    }
    if (argc == 6 && std::strcmp(argv[1], "arpa") == 0) {
        const std::vector<char> text = slurp(argv[2]);
        std::ifstream vf(argv[3]);
        std::vector<std::string> words;
        for (std::string w; std::getline(vf, w);) words.push_back(w);
        std::vector<const char *> vocab;
        for (const std::string &w : words) vocab.push_back(w.c_str());
        const uint32_t flags = uint32_t(std::strtoul(argv[4], nullptr, 10));
        ngpu_arpa *a = nullptr;
        int rc = ngpu_arpa_parse(text.data(), text.size(), vocab.data(), int32_t(vocab.size()), flags, &a);
        ngpu_lm lm;
        if (rc == NGPU_OK) {
            ngpu_ngram_list list;
            float unk = 0;
            rc = ngpu_arpa_list(a, &list, &unk);
            if (rc == NGPU_OK) rc = ngpu::build_trie(&list, int32_t(vocab.size()), unk, flags, &lm, &err);
            ngpu_arpa_free(a);
        }
        return finish(rc, lm, argv[5]);
    }
    std::fprintf(stderr, "usage: build_driver list LIST OUT | arpa TEXT VOCAB FLAGS OUT\n");
    return 2;
}
