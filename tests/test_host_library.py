"""Host side of the C-ABI library: exports, trie construction, numbering, errors.

None of these tests launches a kernel.  ``test_image_walk_matches_oracle``
walks the host copy of the trie image on the CPU, as Algorithm 1 states it, to
check the builder's arrays against the oracle before any GPU is involved.
"""

import ctypes
import os
import re
import struct

import numpy as np
import pytest

import paper_2505_22857_amd as ng
from oracle import Oracle
from synth import generate_model, make_model, tiny_model, uniform_states

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ngpu_lm.h")


@pytest.fixture(scope="module")
def lib():
    return ng.load_library()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ngpu_(?:lm|arpa)_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol(lib):
    decl = declared_functions()
    assert len(decl) >= 10
    for name in decl:
        assert hasattr(lib, name), name
    assert sorted(ng.EXPORTED) == decl


HDR_FMT = "<IiiiqqQQQQQQ11i4x10QQiiQqiiQQ"


def parse_image(img):
    """White-box view of the image (layout of csrc/trie.h)."""
    raw = img.tobytes()
    f = struct.unpack_from(HDR_FMT, raw)
    magic, V, N, R, S, A3 = f[:6]
    o_st, o_ch, o_dw, o_dt, o_arc, total = f[6:12]
    first = list(f[12:23])
    off_order = list(f[23:33])
    off_final, start_state, has_final, o_top, top_begin, delta = f[33:39]
    compact_rank, o_dc, o_db = f[39:42]
    assert struct.calcsize(HDR_FMT) == 264
    assert magic == 0x354D4C4E and total == len(img)
    lo = np.frombuffer(raw, np.int32, 2 * top_begin, o_arc).reshape(top_begin, 2)    # {token, weight bits}
    hi = np.frombuffer(raw, np.int32, 3 * (A3 - top_begin), o_top).reshape(-1, 3)  # {token, weight bits, next}
    arcs = np.concatenate([lo, hi[:, :2]])
    # next state: index + delta below the highest order, stored at it
    to = np.concatenate([np.arange(top_begin, dtype=np.int64) + delta, hi[:, 2]]).astype(np.int32)
    return dict(V=V, N=N, R=R, S=S, A=A3, first=first, off_order=off_order, raw=raw, o_ch=o_ch,
                dense_w=np.frombuffer(raw, np.float32, R * V, o_dw).reshape(R, V),
                dense_to=np.frombuffer(raw, np.int32, R * V, o_dt).reshape(R, V),
                tok=arcs[:, 0].copy(), w=arcs[:, 1].copy().view(np.float32), to=to,
                start_state=start_state,
                final=np.frombuffer(raw, np.float32, S, off_final) if has_final else None,
                compact_rank=compact_rank,
                dense_c=np.frombuffer(raw, np.uint32, R * V, o_dc).reshape(R, V) if o_dc else None,
                dense_base=np.frombuffer(raw, np.int32, R, o_db) if o_dc else None)


@pytest.mark.parametrize("which", ["trigram_v128", "fourgram_200k", "n2", "n10", "bos_eos", "tiny-unk", "n1",
                                   "positive"])
def test_compact_dense_rows(which):
    """The 4-byte dense rows of the register decode: present exactly when V <= 1024,
    every dense weight is negative (sign bit set) and every unigram is listed;
    then the weight is the stored magnitude with the sign bit set, the sign bit
    marks the backed-off entries, and a token's next state is first[1] + v for
    backed-off entries (and row 0), else (orders >= 3) the row's base plus the
    token's rank among the row's own entries, as the 8-byte rows hold it."""
    expect = True
    if which in ("trigram_v128", "fourgram_200k"):
        m = make_model(which)
    elif which == "n2":
        m = generate_model(40, [40, 400], 1.0, seed=1)
    elif which == "n10":
        m = generate_model(16, [16, 120, 200, 200, 180, 160, 140, 120, 100, 80], 1.0, seed=3)
    elif which == "bos_eos":
        m = generate_model(24, [24, 180, 240, 200], 1.0, seed=3, bos_eos=True)
    elif which == "tiny-unk":
        m, expect = tiny_model(9, 3, seed=21, n_unigrams=6), False
    elif which == "n1":
        m, expect = generate_model(40, [40], 1.0, seed=1), False
    else:
        m, expect = generate_model(40, [40, 400], 1.0, seed=1), False
    if which == "positive":   # one weight at +0.0: its sign bit is clear
        order, tokens, W, B = m.to_list()
        W = W.copy()
        W[np.nonzero(order == 2)[0][0]] = 0.0
        lm = ng.NgpuLM(m.vocab_size, m.max_order, order, tokens, W, B, m.unk_logprob)
    else:
        lm = ng.NgpuLM.from_model(m)
    im = parse_image(lm.host_image())
    assert (im["dense_c"] is not None) == expect
    if not expect:
        return
    V, f1 = im["V"], im["first"][1]
    wbits = im["dense_w"].view(np.uint32)
    c = im["dense_c"]
    assert np.array_equal(c | np.uint32(0x80000000), wbits)
    backoff = im["dense_to"] < 0
    assert not backoff[0].any()
    assert np.array_equal(c >> 31 == 1, backoff)
    for u in range(im["R"]):
        own = ~backoff[u]
        nxt = np.full(V, -1, np.int64)
        nxt[~own] = f1 + np.nonzero(~own)[0]
        if im["compact_rank"] and u > 0:
            nxt[own] = im["dense_base"][u] + np.arange(own.sum())
        else:
            nxt[own] = f1 + np.nonzero(own)[0]
        assert np.array_equal(nxt, im["dense_to"][u] & 0x7FFFFFFF), (which, u)


def chain_of(im, s):
    k = 0
    for j in range(1, 10):
        if s >= im["first"][j]:
            k = j
    off = im["o_ch"] + im["off_order"][k] + (s - im["first"][k]) * 16 * max(k, 1)
    row, acc1, acc0, nlev_group = struct.unpack_from("<iffi", im["raw"], off)
    nlev = nlev_group & 0xFFFF
    levels = [struct.unpack_from("<iif", im["raw"], off + 16 * (j + 1)) for j in range(nlev)]
    return k, row, np.float32(acc1), np.float32(acc0), levels


def walk_image(im, s):
    """The query over the image arrays on the CPU: sparse levels, then the dense row."""
    V = im["V"]
    nxt = np.full(V, -1, np.int32)
    sc = np.zeros(V, np.float32)
    k, row, acc1, acc0, levels = chain_of(im, s)
    for b, e, acc in levels:
        toks = im["tok"][b:e]
        unset = nxt[toks] == -1
        sc[toks[unset]] = np.float32(acc) + im["w"][b:e][unset]
        nxt[toks[unset]] = im["to"][b:e][unset]
    unset = nxt == -1
    dt = im["dense_to"][row]
    flag = dt < 0
    acc = np.where(flag, acc0, acc1).astype(np.float32)
    sc[unset] = (acc + im["dense_w"][row])[unset]
    nxt[unset] = (dt & 0x7FFFFFFF)[unset]
    return sc, nxt


@pytest.mark.parametrize("which", ["trigram_v128", "fourgram_200k", "tiny-unk", "n1", "n2", "n10"])
def test_image_walk_matches_oracle(which):
    if which == "trigram_v128":
        m, states = make_model("trigram_v128"), None
    elif which == "fourgram_200k":
        m = make_model("fourgram_200k")
        states = uniform_states(m, 300, seed=2)
    elif which == "tiny-unk":
        m, states = tiny_model(9, 3, seed=21, n_unigrams=6), None
    elif which == "n1":
        m, states = generate_model(40, [40], 1.0, seed=1), None
    elif which == "n2":
        m, states = generate_model(40, [40, 400], 1.0, seed=1), None
    else:
        m = generate_model(16, [16, 120, 200, 200, 180, 160, 140, 120, 100, 80], 1.0, seed=3)
        states = None
    lm = ng.NgpuLM.from_model(m, shuffle_seed=7)
    o = Oracle.from_model(m)
    assert lm.num_states == o.num_states == m.num_states
    if states is None:
        states = np.arange(m.num_states, dtype=np.int32)
    im = parse_image(lm.host_image())
    s32, nx, _ = o.advance(states, nthreads=4)
    for i, s in enumerate(states):
        sc, n = walk_image(im, int(s))
        assert np.array_equal(n, nx[i]), (which, s)
        assert np.array_equal(sc, s32[i]), (which, s)   # same fp32 fold: bit-exact


def test_bos_eos_image_matches_oracle():
    """<s>/</s> models: numbering, rows, start state and final weights vs the oracle."""
    for seed in (3, 7):
        m = generate_model(24, [24, 180, 240, 200], 1.0, seed=seed, bos_eos=True)
        lm = ng.NgpuLM.from_model(m, shuffle_seed=seed)
        o = Oracle.from_model(m)
        assert lm.num_states == o.num_states == m.num_states
        assert lm.start_state == o.start_state == m.start_state
        assert lm.state_context(lm.start_state) == (24,)
        im = parse_image(lm.host_image())
        states = np.arange(m.num_states, dtype=np.int32)
        s32, nx, _ = o.advance(states)
        for s_ in states:
            sc, n = walk_image(im, int(s_))
            assert np.array_equal(n, nx[s_]) and np.array_equal(sc, s32[s_])
        assert np.array_equal(im["final"], o.final(states))      # same fp32 fold: bit-exact


def test_bos_eos_build_errors():
    V = 3
    order = np.array([1, 1, 1, 1, 1, 2, 2], np.int32)
    tokens = np.array([[0, -1], [1, -1], [2, -1], [3, -1], [4, -1], [3, 0], [0, 4]], np.int32)
    W = np.array([-1, -1, -1, -99, -2, -0.5, -0.5], np.float32)
    B = np.zeros(7, np.float32)
    lib = ng.load_library()

    def build(o, t, w, b, flags):
        o, t, w, b = (np.ascontiguousarray(x) for x in (o, t, w, b))
        lst = ng._NgramList(len(o), 2, o.ctypes.data, t.ctypes.data, w.ctypes.data, b.ctypes.data)
        h = ctypes.c_void_p()
        rc = lib.ngpu_lm_build(ctypes.byref(lst), V, float("nan"), flags, ctypes.byref(h))
        if rc == 0:
            lib.ngpu_lm_free(h)
        return rc
    assert build(order, tokens, W, B, 1) == 0
    assert build(order, tokens, W, B, 0) == -2                 # ids V, V+1 without the flag
    bad = tokens.copy(); bad[6] = [4, 0]                       # </s> opening an n-gram
    assert build(order, bad, W, B, 1) == -2
    bad = tokens.copy(); bad[5] = [0, 3]                       # <s> closing an n-gram
    assert build(order, bad, W, B, 1) == -2
    keep = np.array([1, 1, 1, 0, 1, 0, 1], bool)               # no <s> unigram
    assert build(order[keep], tokens[keep], W[keep], B[keep], 1) == -7
    keep = np.array([1, 1, 1, 1, 0, 1, 0], bool)               # no </s> unigram, no <unk>
    assert build(order[keep], tokens[keep], W[keep], B[keep], 1) == -7
    assert build(order, tokens, W, B, 4) == -1                 # unknown flag


def test_numbering_matches_oracle_on_shuffled_lists():
    for idx, key in ((1, "trigram_v128"), (2, "fourgram_200k")):
        m = make_model(key)
        lm = ng.NgpuLM.from_model(m, shuffle_seed=idx)
        o = Oracle.from_model(m, shuffle_seed=idx + 10)
        S = lm.num_states
        ids = range(S) if S < 5000 else np.random.default_rng(0).integers(0, S, 3000)
        for s in ids:
            assert lm.state_context(int(s)) == o.state_context(int(s))


def test_chain_records_and_sparse_rows():
    m = make_model("fourgram_200k")
    lm = ng.NgpuLM.from_model(m)
    o = Oracle.from_model(m)
    im = parse_image(lm.host_image())
    order, tokens, W, B = m.to_list()
    Bd = {tuple(t[:k]): b for k, t, b in zip(order, tokens, B)}
    assert im["R"] == 1 + m.counts[0]
    for s in np.random.default_rng(1).integers(1, im["S"], 400):
        ctx = o.state_context(int(s))
        k, row, acc1, acc0, levels = chain_of(im, int(s))
        assert k == len(ctx) and len(levels) == k - 1
        # dense row = the order-1 ancestor (the context's last token); accumulators are the fp32 fold
        assert row == o.state_of(ctx[-1:])
        acc = np.float32(0.0)
        for j, (b, e, a) in enumerate(levels):
            assert np.float32(a) == acc
            t = im["tok"][b:e]
            assert (np.diff(t) > 0).all() and (b <= e)
            acc = np.float32(acc + np.float32(Bd[ctx[j:]]))
        assert acc1 == acc and acc0 == np.float32(acc + np.float32(Bd[ctx[-1:]]))
    # the dense row of an order-1 state flags exactly the tokens it does not continue with
    u = 5
    flagged = im["dense_to"][u] < 0
    own = {int(t[1]) for k, t in zip(order, tokens) if k == 2 and t[0] == u - 1}
    assert set(np.nonzero(~flagged)[0].tolist()) == own


def _raw_build(V, N, order, tokens, W, B, unk=float("nan"), flags=0):
    lib = ng.load_library()
    order = np.ascontiguousarray(order, np.int32)
    tokens = np.ascontiguousarray(tokens, np.int32)
    W = np.ascontiguousarray(W, np.float32)
    B = np.ascontiguousarray(B, np.float32)
    lst = ng._NgramList(len(order), N, order.ctypes.data, tokens.ctypes.data, W.ctypes.data, B.ctypes.data)
    h = ctypes.c_void_p()
    rc = lib.ngpu_lm_build(ctypes.byref(lst), V, unk, flags, ctypes.byref(h))
    if rc == 0:
        lib.ngpu_lm_free(h)
    return rc, lib.ngpu_lm_last_error().decode()


def _fig1():
    order = np.array([1, 1, 1, 2, 2, 3], np.int32)
    tokens = np.array([[0, -1, -1], [1, -1, -1], [2, -1, -1], [0, 1, -1], [1, 2, -1], [0, 1, 2]], np.int32)
    W = np.array([-1, -1, -1, -0.5, -0.5, -0.1], np.float32)
    B = np.array([-0.3, -0.3, -0.3, -0.2, -0.2, 0], np.float32)
    return order, tokens, W, B


def test_build_error_codes():
    o, t, W, B = _fig1()
    assert _raw_build(3, 3, o, t, W, B)[0] == 0
    assert _raw_build(3, 3, np.append(o, 2), np.vstack([t, t[3]]), np.append(W, 0), np.append(B, 0))[0] == -4
    bad = t.copy(); bad[1, 0] = 3
    assert _raw_build(3, 3, o, bad, W, B)[0] == -2
    bad = o.copy(); bad[0] = 4
    assert _raw_build(3, 3, bad, t, W, B)[0] == -3
    assert _raw_build(3, 11, o, np.pad(t, ((0, 0), (0, 8)), constant_values=-1), W, B)[0] == -3
    # trigram (0 1 2) without its prefix (0 1)
    keep = np.array([1, 1, 1, 0, 1, 1], bool)
    assert _raw_build(3, 3, o[keep], t[keep], W[keep], B[keep])[0] == -5
    # trigram (0 1 2) without its suffix (1 2)
    keep = np.array([1, 1, 1, 1, 0, 1], bool)
    assert _raw_build(3, 3, o[keep], t[keep], W[keep], B[keep])[0] == -6
    # a token with no unigram: error without <unk>, fine with it
    assert _raw_build(4, 3, o, t, W, B)[0] == -7
    assert _raw_build(4, 3, o, t, W, B, unk=-5.0)[0] == 0
    Wn = W.copy(); Wn[2] = np.nan
    assert _raw_build(3, 3, o, t, Wn, B)[0] == -10
    assert _raw_build(ng.MAX_VOCAB + 1, 3, o, t, W, B)[0] == -11
    assert _raw_build(3, 3, o, t, W, B, flags=4)[0] == -1          # unknown flag
    assert _raw_build(3, 3, o, t, W, B, flags=2)[0] == 0           # closure repair of a closed list


def test_queries_before_upload_fail_cleanly():
    m = make_model("trigram_v128")
    lm = ng.NgpuLM.from_model(m)
    lib = ng.load_library()
    assert lib.ngpu_lm_advance(lm._h, None, 4, None, None, None) == -8
    assert lib.ngpu_lm_fused_greedy_step(lm._h, None, 4, 129, 0, 0.5, None, None, None, None) == -8
    n = ctypes.c_int64()
    assert lib.ngpu_lm_check_states(lm._h, None, ctypes.byref(n)) == -8
    assert "not uploaded" in lib.ngpu_lm_last_error().decode()


def test_query_bytes():
    m = make_model("fourgram_200k")
    lm = ng.NgpuLM.from_model(m)
    V = m.vocab_size
    hbm, tot = lm.query_bytes(np.zeros(3, np.int32))
    assert hbm == 3 * (8 * V + 16) and tot == hbm + 3 * 8 * V
    im = parse_image(lm.host_image())
    s = m.state_offset(3) + 5                      # an order-3 state: two sparse levels
    k, row, acc1, acc0, levels = chain_of(im, s)
    arcs = sum(e - b for b, e, _ in levels)
    hbm, tot = lm.query_bytes(np.array([s], np.int32))
    assert hbm == 8 * V + 16 * 3 + 12 * arcs
    assert tot == hbm + 8 * V
    with pytest.raises(ng.NgpuError):
        lm.query_bytes(np.array([m.num_states], np.int32))
