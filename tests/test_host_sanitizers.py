"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer.

The trie builder and the ARPA reader (host C++ of the library) and the oracle
(C) are compiled with gcc/g++ and ``-fsanitize=address,undefined`` into small
drivers (``tests/sanitize/``) and run on generated models, sentence-marker
models, malformed lists and ARPA text.  Any sanitizer report aborts the driver
(``-fno-sanitize-recover=all``); the outputs must also equal those of the
normal builds byte for byte: the library's host image and error codes, and the
oracle's advance, decodes, top-k and final weights.
"""

import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
import paper_2505_22857_amd as ng
from oracle import MODE_AED, MODE_CTC, MODE_PLAIN, Oracle
from synth import (asr_logprobs, bpe_like_vocab, generate_model, make_model, pruned_list, tiny_model,
                   write_arpa)

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2505_22857_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1",
       "-ffp-contract=off"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")


def _compile(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        if "asan" in r.stderr.lower() or "ubsan" in r.stderr.lower():
            pytest.skip("sanitizer runtime not available: " + r.stderr[-300:])
        raise AssertionError("compile failed:\n" + r.stderr[-3000:])


@pytest.fixture(scope="module")
def drivers(tmp_path_factory):
    if shutil.which("g++") is None or shutil.which("gcc") is None:
        pytest.skip("gcc/g++ not available")
    d = tmp_path_factory.mktemp("san")
    bd, od = str(d / "build_driver"), str(d / "oracle_driver")
    _compile(["g++", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "include"), "-I", CSRC,
              os.path.join(CSRC, "trie_build.cpp"), os.path.join(CSRC, "arpa.cpp"),
              os.path.join(HERE, "sanitize", "build_driver.cpp"), "-o", bd])
    _compile(["gcc", *SAN, "-pthread", os.path.join(ROOT, "oracle", "oracle.c"),
              os.path.join(HERE, "sanitize", "oracle_driver.c"), "-o", od, "-lm"])
    return bd, od, d


def _write_list(path, V, N, order, tokens, W, B, unk, flags):
    with open(path, "wb") as f:
        f.write(np.array([V, N], np.int32).tobytes())
        f.write(np.array([len(order)], np.int64).tobytes())
        f.write(np.array([unk], np.float32).tobytes())
        f.write(np.array([flags], np.uint32).tobytes())
        f.write(np.ascontiguousarray(order, np.int32).tobytes())
        f.write(np.ascontiguousarray(tokens, np.int32).reshape(-1).tobytes())
        f.write(np.ascontiguousarray(W, np.float32).tobytes())
        f.write(np.ascontiguousarray(B, np.float32).tobytes())


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True, env=ENV, timeout=300)
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    assert r.returncode == 0, f"rc {r.returncode}\n{r.stderr[-4000:]}"
    return r.stdout


def _models():
    return {
        "trigram_v128": make_model("trigram_v128"),
        "unk": tiny_model(9, 3, seed=21, n_unigrams=6),
        "bos_eos": generate_model(40, [40, 300, 500, 300], 1.0, seed=5, bos_eos=True),
        "unigram": generate_model(17, [17], 1.0, seed=6),
    }


@pytest.mark.parametrize("name", ["trigram_v128", "unk", "bos_eos", "unigram"])
def test_builder_clean_and_identical(drivers, name):
    bd, _, d = drivers
    m = _models()[name]
    o, t, W, B = m.to_list(shuffle_seed=3)
    flags = 1 if m.bos_eos else 0
    lst, img = str(d / f"{name}.list"), str(d / f"{name}.img")
    _write_list(lst, m.vocab_size, m.max_order, o, t, W, B, m.unk_logprob, flags)
    assert _run([bd, "list", lst, img]).split() == ["rc", "0"]
    ref = ng.NgpuLM(m.vocab_size, m.max_order, o, t, W, B, m.unk_logprob, bos_eos=m.bos_eos).host_image()
    assert np.array_equal(np.fromfile(img, np.uint8), ref)


@pytest.mark.parametrize("seed", [6, 7])
def test_builder_repair_clean_and_identical(drivers, seed):
    """A pruned list built with closure repair (flag 2)."""
    bd, _, d = drivers
    m = generate_model(8, [8, 40, 90, 100], 1.0, seed=seed)
    o, t, W, B = pruned_list(m, 0.35, seed=seed + 100)
    lst, img = str(d / f"pruned{seed}.list"), str(d / f"pruned{seed}.img")
    _write_list(lst, 8, 4, o, t, W, B, m.unk_logprob, 2)
    assert _run([bd, "list", lst, img]).split() == ["rc", "0"]
    ref = ng.NgpuLM(8, 4, o, t, W, B, m.unk_logprob, repair=True).host_image()
    assert np.array_equal(np.fromfile(img, np.uint8), ref)


@pytest.mark.parametrize("seed", [6, 7])
def test_oracle_repair_clean_and_identical(drivers, seed):
    _, od, d = drivers
    m = generate_model(8, [8, 40, 90, 100], 1.0, seed=seed)
    o, t, W, B = pruned_list(m, 0.35, seed=seed + 100)
    lst, out = str(d / f"orep{seed}.list"), str(d / f"orep{seed}.out")
    _write_list(lst, 8, 4, o, t, W, B, m.unk_logprob, 0)
    _run([od, "repair", lst, out])
    ro, rt, rW, rB = oracle.repair_list(8, 4, o, t, W, B, m.unk_logprob)
    want = (np.array([len(ro)], np.int64).tobytes() + ro.astype(np.int32).tobytes() + rt.astype(np.int32).tobytes()
            + rW.astype(np.float32).tobytes() + rB.astype(np.float32).tobytes())
    assert open(out, "rb").read() == want


def _broken_lists():
    m = tiny_model(9, 3, seed=21, n_unigrams=9)
    o, t, W, B = m.to_list()
    out = {}
    dup = np.concatenate([np.arange(len(o)), [len(o) - 1]])
    out["duplicate"] = (o[dup], t[dup], W[dup], B[dup])
    hi = np.flatnonzero(o == 3)[0]
    bi = np.array([i for i in range(len(o)) if o[i] == 2 and tuple(t[i, :2]) == tuple(t[hi, :2])])
    keep = np.setdiff1d(np.arange(len(o)), bi)
    out["missing_prefix"] = (o[keep], t[keep], W[keep], B[keep])
    t2 = t.copy()
    t2[0, 0] = 9
    out["token_range"] = (o, t2, W, B)
    o2 = o.copy()
    o2[0] = 4
    out["order_range"] = (o2, t, W, B)
    W2 = W.copy()
    W2[3] = np.inf
    out["nonfinite"] = (o, t, W2, B)
    return m, out


@pytest.mark.parametrize("case", ["duplicate", "missing_prefix", "token_range", "order_range", "nonfinite"])
def test_builder_malformed_lists(drivers, case):
    bd, _, d = drivers
    m, lists = _broken_lists()
    o, t, W, B = lists[case]
    lst = str(d / f"bad_{case}.list")
    _write_list(lst, m.vocab_size, m.max_order, o, t, W, B, m.unk_logprob, 0)
    rc = int(_run([bd, "list", lst, str(d / "bad.img")]).split()[1])
    with pytest.raises(ng.NgpuError) as e:
        ng.NgpuLM(m.vocab_size, m.max_order, o, t, W, B, m.unk_logprob)
    assert rc == e.value.code and rc < 0


@pytest.mark.parametrize("bos_eos", [False, True])
def test_arpa_reader_clean_and_identical(drivers, bos_eos):
    bd, _, d = drivers
    m = generate_model(40, [40, 300, 500, 300], 1.0, seed=5, bos_eos=True)
    voc = bpe_like_vocab(40)
    txt, vf, img = d / "m.arpa", d / "vocab.txt", str(d / f"arpa{int(bos_eos)}.img")
    txt.write_text(write_arpa(m, voc))
    vf.write_text("\n".join(voc) + "\n")
    assert _run([bd, "arpa", str(txt), str(vf), str(int(bos_eos)), img]).split() == ["rc", "0"]
    N, o, t, W, B, unk = ng.parse_arpa(txt.read_text(), voc, bos_eos=bos_eos)
    ref = ng.NgpuLM(40, N, o, t, W, B, unk, bos_eos=bos_eos).host_image()
    assert np.array_equal(np.fromfile(img, np.uint8), ref)


@pytest.mark.parametrize("text", ["no header at all", "\\data\\\nngram 1=2\n\n\\1-grams:\n-1\tw0\n", "\\data\\\n"])
def test_arpa_reader_malformed_text(drivers, text):
    bd, _, d = drivers
    voc = bpe_like_vocab(40)
    txt, vf = d / "bad.arpa", d / "vocab.txt"
    txt.write_text(text)
    vf.write_text("\n".join(voc) + "\n")
    rc = int(_run([bd, "arpa", str(txt), str(vf), "0", str(d / "bad.img")]).split()[1])
    with pytest.raises(ng.NgpuError) as e:
        ng.parse_arpa(text, voc)
    assert rc == e.value.code and rc < 0


@pytest.mark.parametrize("name", ["trigram_v128", "bos_eos"])
def test_oracle_clean_and_identical(drivers, name):
    _, od, d = drivers
    m = _models()[name]
    o, t, W, B = m.to_list()
    flags = 1 if m.bos_eos else 0
    V, K = m.vocab_size, 5
    lst, af, out = str(d / f"o_{name}.list"), str(d / f"o_{name}.asr"), str(d / f"o_{name}.out")
    _write_list(lst, V, m.max_order, o, t, W, B, m.unk_logprob, flags)
    Bq, T = 4, 30
    asr = asr_logprobs((Bq, T, V + 1), seed=7, blank_boost=1.0)
    with open(af, "wb") as f:
        f.write(np.array([Bq, T], np.int64).tobytes())
        f.write(asr.tobytes())
    _run([od, lst, af, str(K), out])
    got = open(out, "rb").read()
    ref = Oracle.from_model(m)
    S = ref.num_states
    parts = []
    s32, nx, _ = ref.advance(np.arange(S, dtype=np.int32), nthreads=2)
    parts += [s32.astype(np.float32).tobytes(), nx.astype(np.int32).tobytes()]
    for mode in (MODE_PLAIN, MODE_CTC) + ((MODE_AED,) if m.bos_eos else ()):
        starts = np.full(Bq, ref.start_state if mode == MODE_AED else 0, np.int32)
        lab, sts = ref.decode(asr, mode, 0.5, starts, nthreads=2)
        parts += [lab.astype(np.int32).tobytes(), sts.astype(np.int32).tobytes()]
    tt, ts, tn = ref.fused_topk(np.ascontiguousarray(asr[:, 0, :]), 0.7, K, (np.arange(Bq) % S).astype(np.int32))
    parts += [tt.astype(np.int32).tobytes(), ts.astype(np.float32).tobytes(), tn.astype(np.int32).tobytes()]
    if m.bos_eos:
        parts.append(ref.final(np.arange(S, dtype=np.int32)).astype(np.float32).tobytes())
    assert got == b"".join(parts)
