"""Closure repair of pruned n-gram lists (NGPU_BUILD_REPAIR_CLOSURE), host side.

The library's repair (in the trie builder) must give the same trie, byte for
byte, as the list the oracle's own repair produces (``oracle.repair_list``,
pinned against brute force on histories in test_oracle_pins.py): same added
n-grams, same weights, same state numbering.
"""

import numpy as np
import pytest

import oracle
import paper_2505_22857_amd as ng
from synth import (bpe_like_vocab, generate_model, make_model, pruned_list, tiny_model,
                   write_arpa_list)


def _cases():
    return {
        "V8N4 seed 6": (generate_model(8, [8, 40, 90, 100], 1.0, seed=6), 0.35, 0),
        "V8N4 seed 7": (generate_model(8, [8, 40, 90, 100], 1.0, seed=7), 0.35, 0),
        "sentence markers": (generate_model(20, [20, 150, 200, 150], 1.0, seed=3, bos_eos=True), 0.3, 0),
        "unk, a unigram dropped": (tiny_model(9, 3, seed=21, n_unigrams=8), 0.3, 1),
        "4-gram 200k": (make_model("fourgram_200k"), 0.2, 0),
    }


@pytest.mark.parametrize("name", sorted(_cases()))
def test_library_repair_equals_oracle_repair(name):
    m, drop, du = _cases()[name]
    V, N = m.vocab_size, m.max_order
    o, t, W, B = pruned_list(m, drop, seed=11, drop_unigrams=du)
    with pytest.raises(ng.NgpuError) as e:
        ng.NgpuLM(V, N, o, t, W, B, m.unk_logprob, bos_eos=m.bos_eos)
    assert e.value.code in (-5, -6)          # NGPU_E_MISSING_PREFIX / NGPU_E_MISSING_SUFFIX
    lib = ng.NgpuLM(V, N, o, t, W, B, m.unk_logprob, bos_eos=m.bos_eos, repair=True)
    R = oracle.repair_list(V, N, o, t, W, B, m.unk_logprob, bos_eos=m.bos_eos)
    ref = ng.NgpuLM(V, N, *R, m.unk_logprob, bos_eos=m.bos_eos)
    assert lib.num_states == ref.num_states and len(R[0]) > len(o)
    assert np.array_equal(lib.host_image(), ref.host_image())


def test_repair_leaves_closed_lists_alone():
    for m in (make_model("trigram_v128"), generate_model(20, [20, 150, 200, 150], 1.0, seed=3, bos_eos=True)):
        a = ng.NgpuLM.from_model(m)
        b = ng.NgpuLM(m.vocab_size, m.max_order, *m.to_list(), m.unk_logprob, bos_eos=m.bos_eos, repair=True)
        assert np.array_equal(a.host_image(), b.host_image())


def test_repair_needs_unk_for_a_missing_unigram():
    m = generate_model(8, [8, 40, 90], 1.0, seed=2)
    o, t, W, B = m.to_list()
    v = int(t[np.flatnonzero(o == 2)[0], 1])       # a token that ends a bigram
    keep = ~((o == 1) & (t[:, 0] == v))
    with pytest.raises(ng.NgpuError) as e:
        ng.NgpuLM(8, 3, o[keep], t[keep], W[keep], B[keep], float("nan"), repair=True)
    assert e.value.code == -7                     # NGPU_E_MISSING_UNIGRAM
    with pytest.raises(oracle.OracleError):
        oracle.repair_list(8, 3, o[keep], t[keep], W[keep], B[keep], float("nan"))
    # with an <unk> weight the unigram is added with it
    lib = ng.NgpuLM(8, 3, o[keep], t[keep], W[keep], B[keep], -9.5, repair=True)
    R = oracle.repair_list(8, 3, o[keep], t[keep], W[keep], B[keep], -9.5)
    row = [i for i in range(len(R[0])) if R[0][i] == 1 and R[1][i, 0] == v]
    assert len(row) == 1 and R[2][row[0]] == np.float32(-9.5)
    assert np.array_equal(lib.host_image(), ng.NgpuLM(8, 3, *R, -9.5).host_image())


def test_repair_of_a_pruned_arpa_file():
    m = generate_model(40, [40, 300, 500, 300], 1.0, seed=5, bos_eos=True)
    o, t, W, B = pruned_list(m, 0.3, seed=12)
    voc = bpe_like_vocab(40)
    txt = write_arpa_list(40, 4, o, t, W, B, m.unk_logprob, voc, bos_eos=True)
    N, po, pt, pW, pB, unk = ng.parse_arpa(txt, voc, bos_eos=True)
    a = ng.NgpuLM(40, N, po, pt, pW, pB, unk, bos_eos=True, repair=True)
    b = ng.NgpuLM(40, 4, o, t, W, B, m.unk_logprob, bos_eos=True, repair=True)
    assert np.array_equal(a.host_image(), b.host_image())
