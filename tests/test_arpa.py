"""The library's ARPA reader (host only).

Files written from generated models (synth.write_arpa, base-10 logarithms with
17 significant digits) must read back to the same n-gram list; a trie built
from the parsed list must be byte-identical to one built from the list.  A
hand-written file pins the log10 -> ln conversion and the special words.
"""

import math

import numpy as np
import pytest

import paper_2505_22857_amd as ng
from synth import bpe_like_vocab, generate_model, make_model, tiny_model, write_arpa


def sorted_list(order, tokens, W, B):
    key = np.lexsort(np.column_stack([tokens, order]).T[::-1])
    return order[key], tokens[key], W[key], B[key]


def test_round_trip_plain_model_is_exact():
    m = make_model("trigram_v128")
    voc = bpe_like_vocab(m.vocab_size)
    N, o, t, W, B, unk = ng.parse_arpa(write_arpa(m, voc), voc)
    o2, t2, W2, B2 = m.to_list()
    assert N == m.max_order and np.isnan(unk)
    for a, b in zip(sorted_list(o, t, W, B), sorted_list(o2, t2, W2, B2)):
        assert np.array_equal(a, b)
    built = ng.NgpuLM(m.vocab_size, N, o, t, W, B, unk)
    direct = ng.NgpuLM.from_model(m)
    assert np.array_equal(built.host_image(), direct.host_image())


def test_round_trip_with_unk():
    m = tiny_model(9, 3, seed=21, n_unigrams=6)
    voc = bpe_like_vocab(9)
    N, o, t, W, B, unk = ng.parse_arpa(write_arpa(m, voc), voc)
    assert unk == np.float32(m.unk_logprob)
    assert len(o) == m.num_ngrams and not (t == -2).any()
    built = ng.NgpuLM(9, N, o, t, W, B, unk)
    assert np.array_equal(built.host_image(), ng.NgpuLM.from_model(m).host_image())


def test_sentence_markers_kept_or_dropped():
    m = generate_model(20, [20, 150, 200, 150], 1.0, seed=3, bos_eos=True)
    voc = bpe_like_vocab(20)
    txt = write_arpa(m, voc)
    N, o, t, W, B, unk = ng.parse_arpa(txt, voc, bos_eos=True)
    o2, t2, W2, B2 = m.to_list()
    for a, b in zip(sorted_list(o, t, W, B), sorted_list(o2, t2, W2, B2)):
        assert np.array_equal(a, b)
    built = ng.NgpuLM(20, N, o, t, W, B, unk, bos_eos=True)
    assert np.array_equal(built.host_image(), ng.NgpuLM.from_model(m).host_image())
    # without the flag every n-gram holding <s> or </s> is dropped; the rest stays closed
    N, o, t, W, B, unk = ng.parse_arpa(txt, voc)
    special = ((t2 == 20) | (t2 == 21)).any(axis=1)
    assert len(o) == int((~special).sum())
    lm = ng.NgpuLM(20, N, o, t, W, B, unk)
    assert lm.num_states == 1 + int(((o2 < N) & ~special).sum())


FIG1 = """
\\data\\
ngram 1=8
ngram 2=3
ngram 3=1

\\1-grams:
-0.4342944819032518\tthe\t-0.21714724095162590
-0.8685889638065036\tcat\t-0.13028834457097554
-0.8685889638065036\tsat\t-0.13028834457097554
-99\t<s>\t-0.3
-0.8685889638065036\t</s>
-2.0\t<unk>\t0
-0.8685889638065036\ton
-0.8685889638065036\tmat

\\2-grams:
-0.30400613733227626\tthe cat\t-0.08685889638065036
-0.1\t<s> the\t-0.1
-0.2\tmat </s>

\\3-grams:
-0.021714724095162591\t<s> the cat

\\end\\
"""


def test_hand_written_file():
    voc = ["the", "cat", "sat", "on", "mat"]
    ln10 = math.log(10.0)
    N, o, t, W, B, unk = ng.parse_arpa(FIG1, voc, bos_eos=True)
    assert N == 3 and unk == np.float32(-2.0 * ln10)
    rows = {tuple(int(x) for x in tt[:k]): (w, b) for k, tt, w, b in zip(o, t, W, B)}
    assert rows[(0,)] == (np.float32(-1.0), np.float32(-0.5))
    assert rows[(1,)] == (np.float32(-2.0), np.float32(-0.3))
    assert rows[(0, 1)] == (np.float32(-0.7), np.float32(-0.2))
    assert rows[(5, 0, 1)][0] == np.float32(-0.05)
    assert rows[(6,)][0] == np.float32(-2.0) and rows[(4, 6)][0] == np.float32(-0.2 * ln10)
    assert rows[(5,)][0] == np.float32(-99 * ln10)
    lm = ng.NgpuLM(5, N, o, t, W, B, unk, bos_eos=True)
    assert lm.state_context(lm.start_state) == (5,)
    # without sentence markers: <s>, </s> and the n-grams holding them go
    N, o, t, W, B, unk = ng.parse_arpa(FIG1, voc)
    assert len(o) == 6 and not ((t >= 5).any())


@pytest.mark.parametrize("text,code", [
    (FIG1.replace("\tcat\t", "\tdog\t"), -2),                       # unknown word
    (FIG1.replace("ngram 2=3", "ngram 2=4"), -1),                    # count mismatch
    (FIG1.replace("\\end\\", ""), -1),                               # no end marker
    (FIG1.replace("-0.1\t<s> the\t-0.1", "-0.1\t<s> the cat on\t-0.1"), -1),   # too many fields
    (FIG1.replace("-2.0\t<unk>", "x2.0\t<unk>"), -10),               # unreadable weight
    (FIG1.replace("\\2-grams:", "\\3-grams:"), -1),                  # sections out of order
    ("no header at all", -1),
])
def test_parse_errors(text, code):
    with pytest.raises(ng.NgpuError) as e:
        ng.parse_arpa(text, ["the", "cat", "sat", "on", "mat"], bos_eos=True)
    assert e.value.code == code


def test_vocabulary_errors():
    with pytest.raises(ng.NgpuError):
        ng.parse_arpa(FIG1, ["the", "cat", "sat", "on", "the"])      # duplicate word
    with pytest.raises(ng.NgpuError):
        ng.parse_arpa(FIG1, ["the", "cat", "sat", "on", "<s>"])      # special word in the vocabulary
