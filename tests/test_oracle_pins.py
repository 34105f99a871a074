"""Pins of the CPU oracle against what the paper and the mathematics fix.

No implementation of the method exists to compare with, so the oracle is tied
down by: hand-derived values on the Figure 1 sentence (tests/golden), the
backoff rule restated on raw histories (brute force on tiny models), per-context
normalisation of models built normalised, the textbook reductions (unigram
model, bigram backoff, lambda = 0 fusion, greedy CTC), structural invariants of
the suffix graph, and the fp32 summation error bound.  The last test plants
mistakes in copies of the oracle and checks that some pin catches each one.
"""

import itertools
import json
from fractions import Fraction
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from oracle import MODE_AED, MODE_CTC, MODE_PLAIN, MODE_TRANSDUCER, Oracle
from oracle.bruteforce import BruteForce
from synth import (asr_logprobs, generate_model, make_model, phrase_states, pruned_list, state_ids_of,
                   tiny_model,
                   uniform_states)

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = os.path.join(HERE, "golden")


def fig1_list():
    with open(os.path.join(GOLDEN, "fig1_trigram.json")) as f:
        fx = json.load(f)
    N = fx["max_order"]
    ng = fx["ngrams"]
    order = np.array([len(g[0]) for g in ng], np.int32)
    tokens = np.full((len(ng), N), -1, np.int32)
    for i, g in enumerate(ng):
        tokens[i, :len(g[0])] = g[0]
    W = np.array([g[1] for g in ng], np.float32)
    B = np.array([g[2] for g in ng], np.float32)
    return fx, (len(fx["vocab"]), N, order, tokens, W, B)


# ---------------------------------------------------------------- pin checks
# Each takes the oracle library path so that the planted-mistake test can run
# the same checks against a mutated oracle.

def check_worked_example(lib_path):
    fx, lst = fig1_list()
    o = Oracle(*lst, lib_path=lib_path)
    assert o.num_states == len(fx["state_contexts"])
    for s, ctx in enumerate(fx["state_contexts"]):
        assert o.state_context(s) == tuple(ctx)
    for s, row in fx["rows"].items():
        s32, nx, s64 = o.advance(np.array([int(s)], np.int32), want64=True)
        np.testing.assert_allclose(s64[0], row["scores"], atol=1e-6)
        np.testing.assert_allclose(s32[0], row["scores"], atol=1e-6)
        assert nx[0].tolist() == row["next"]
    st, tot = 0, 0.0
    sent = fx["sentence"]
    for tok, exp_state, exp_score in zip(sent["tokens"], sent["states"], sent["scores"]):
        s32, nx, s64 = o.advance(np.array([st], np.int32), want64=True)
        assert abs(s64[0, tok] - exp_score) < 1e-6
        tot += s64[0, tok]
        st = int(nx[0, tok])
        assert st == exp_state
    assert abs(tot - sent["total"]) < 1e-5


def check_bruteforce_tiny(lib_path, seeds=(0, 1, 2, 3), max_hist_extra=1):
    for seed in seeds:
        V = 4 + seed % 3
        N = 2 + seed % 3
        model = tiny_model(V, N, seed=100 + seed, fill=0.5)
        o = Oracle.from_model(model, lib_path=lib_path, shuffle_seed=seed)
        bf = BruteForce.from_model(model)
        S = o.num_states
        rows = o.advance(np.arange(S, dtype=np.int32), want64=True)
        s32, nx, s64 = rows
        ctx_of = [o.state_context(s) for s in range(S)]
        for L in range(0, N + max_hist_extra):
            for h in itertools.product(range(V), repeat=L):
                # feed the history from the empty context through the oracle's next states
                st = 0
                for t in h:
                    st = int(nx[st, t])
                assert ctx_of[st] == bf.state_context(h), (seed, h)
                for v in range(V):
                    assert abs(s64[st, v] - bf.score(h, v)) < 1e-9, (seed, h, v)
                    assert ctx_of[int(nx[st, v])] == bf.state_context(h + (v,)), (seed, h, v)


def check_normalisation(lib_path, model, states, tol=1e-5):
    o = Oracle.from_model(model, lib_path=lib_path)
    s32, nx, s64 = o.advance(states, nthreads=8, want64=True)
    tot = np.exp(s64).sum(axis=1)
    assert np.abs(tot - 1.0).max() < tol, np.abs(tot - 1.0).max()
    tot32 = np.exp(s32.astype(np.float64)).sum(axis=1)
    assert np.abs(tot32 - 1.0).max() < tol


def check_lambda_zero_and_ties(lib_path):
    model = tiny_model(7, 3, seed=11)
    o = Oracle.from_model(model, lib_path=lib_path)
    rng = np.random.default_rng(5)
    S = o.num_states
    states = rng.integers(0, S, 64).astype(np.int32)
    asr = rng.standard_normal((64, 7)).astype(np.float32)
    asr[:8] = 0.25                                       # full ties: lowest index wins
    asr[8:16, 2] = asr[8:16, 5] = 9.0                     # two-way ties
    st = states.copy()
    tok = o.greedy_step(asr, MODE_PLAIN, 0.0, st)
    exp = np.argmax(asr, axis=1)                         # numpy: first maximal index
    assert tok.tolist() == exp.tolist()
    _, nx, _ = o.advance(states)
    assert st.tolist() == nx[np.arange(64), exp].tolist()


def check_ctc_rules(lib_path):
    fx, lst = fig1_list()
    o = Oracle(*lst, lib_path=lib_path)
    V = 5
    lam = 10.0
    # frame 0: raw ASR prefers 'cat' (1) a little, LM from the root prefers 'the' (0)
    f0 = np.array([-1.2, -1.0, -3.0, -3.0, -3.0, -4.0], np.float32)
    # frame 1: 'the' wins raw and equals the previous label -> kept, no advance
    f1 = np.array([-0.1, -3.0, -3.0, -3.0, -3.0, -4.0], np.float32)
    # frame 2: blank wins raw -> kept, no advance
    f2 = np.array([-3.0, -3.0, -3.0, -3.0, -3.0, -0.1], np.float32)
    # frame 3: 'on' wins raw; fused over tokens other than the previous label (blank here)
    f3 = np.array([-3.0, -3.0, -3.0, -0.5, -3.0, -4.0], np.float32)
    asr = np.stack([f0, f1, f2, f3])[None]
    labels, states = o.decode(asr, MODE_CTC, lam)
    # frame 0 from the root: fused(v) = asr + 10*unigram -> 'the' (-1.2-10) beats 'cat' (-1.0-20)
    assert labels[0].tolist()[:3] == [0, 0, V]
    assert states[0].tolist()[:3] == [1, 1, 1]
    # frame 3 at state 1 'the': fused = asr + 10*lm; lm row [-1.5,-0.7,-2.5,-2.5,-0.9]
    row = np.array([-1.5, -0.7, -2.5, -2.5, -0.9]) * lam + f3[:V]
    assert labels[0, 3] == int(np.argmax(row)) == 1
    assert states[0, 3] == 6
    # the repeat rule excludes the previous label from stage 2: previous 'cat'
    st = np.array([6], np.int32)
    prev = np.array([1], np.int32)
    f = np.array([[-3.0, -0.9, -0.5, -3.0, -3.0, -4.0]], np.float32)   # 'sat' raw winner
    f[0, 1] = -0.6                                                      # repeat close behind
    tok = o.greedy_step(f, MODE_CTC, lam, st, prev)
    assert tok[0] == 2 and st[0] == 8 and prev[0] == 2
    # transducer: blank kept, otherwise fused argmax over all V
    st = np.array([0], np.int32)
    tok = o.greedy_step(np.array([[-3, -3, -3, -3, -3, -0.1]], np.float32), MODE_TRANSDUCER, lam, st)
    assert tok[0] == V and st[0] == 0
    tok = o.greedy_step(np.array([[-1.2, -1.0, -3, -3, -3, -4]], np.float32), MODE_TRANSDUCER, lam, st)
    assert tok[0] == 0 and st[0] == 1


def check_repair(lib_path, seeds=(6, 7)):
    """Closure repair of pruned lists: the repaired list is closed, adds only
    rows with backoff 0, and its state walk scores every token after every
    history exactly as the backoff rule does on the pruned list (brute force
    on histories); its states are the longest listed contexts of the repaired
    list."""
    for seed in seeds:
        V, N = 8, 4
        m = generate_model(V, [V, 40, 90, 100], 1.0, seed=seed)
        o, t, W, B = pruned_list(m, 0.35, seed=seed + 100)
        ro, rt, rW, rB = oracle.repair_list(V, N, o, t, W, B, m.unk_logprob, lib_path=lib_path)
        rows = {tuple(int(x) for x in rt[i, :ro[i]]): (rW[i], rB[i]) for i in range(len(ro))}
        given = {tuple(int(x) for x in t[i, :o[i]]): (W[i], B[i]) for i in range(len(o))}
        assert len(rows) == len(ro)
        for g, wb in given.items():
            assert rows[g] == wb
        for g, (w, b) in rows.items():
            if g not in given:
                assert b == 0.0 and np.isfinite(w)
            if len(g) >= 2:
                assert g[:-1] in rows and g[1:] in rows
        bf = BruteForce(V, N, o, t, W, B, m.unk_logprob)
        bf_rep = BruteForce(V, N, ro, rt, rW, rB, m.unk_logprob)
        orc = Oracle(V, N, ro, rt, rW, rB, m.unk_logprob, lib_path=lib_path)
        level = [((), 0)]
        for L in range(N + 1):
            sts = np.array([st for _, st in level], np.int32)
            _, nx, s64 = orc.advance(sts, want64=True)
            nxt = []
            for i, (h, st) in enumerate(level):
                assert orc.state_context(st) == bf_rep.state_context(h)
                for v in range(V):
                    assert abs(s64[i, v] - bf.score(h, v)) < 1e-5, (seed, h, v)
                    if L < N:
                        nxt.append((h + (v,), int(nx[i, v])))
            level = nxt


def check_generator_ids(lib_path):
    model = make_model("trigram_v128")
    o = Oracle.from_model(model, lib_path=lib_path, shuffle_seed=3)
    N = model.max_order
    for k in range(1, N):
        toks = model.level_tokens(k)
        ids = state_ids_of(model, toks)
        for i in range(0, len(toks), max(1, len(toks) // 50)):
            assert o.state_of(toks[i]) == ids[i]
            assert o.state_context(int(ids[i])) == tuple(int(t) for t in toks[i])


# ---------------------------------------------------------------- the tests

def test_worked_example_fig1(oracle_lib):
    check_worked_example(oracle.LIB_PATH)


def test_bruteforce_history_recursion_tiny(oracle_lib):
    check_bruteforce_tiny(oracle.LIB_PATH, seeds=range(6))


def test_bruteforce_trigram_v128_sampled_histories(oracle_lib):
    model = make_model("trigram_v128")
    o = Oracle.from_model(model)
    bf = BruteForce.from_model(model)
    rng = np.random.default_rng(7)
    S = o.num_states
    s32, nx, s64 = o.advance(np.arange(S, dtype=np.int32), want64=True)
    for _ in range(3000):
        L = int(rng.integers(0, 6))
        # histories biased toward listed n-grams so deep states are exercised
        h = []
        st = 0
        for _ in range(L):
            v = int(np.argmax(s64[st] + rng.gumbel(size=model.vocab_size)))
            h.append(v)
            st = int(nx[st, v])
        assert o.state_context(st) == bf.state_context(h)
        v = int(rng.integers(0, model.vocab_size))
        assert abs(s64[st, v] - bf.score(h, v)) < 1e-9


def test_normalisation_trigram_v128_all_states(oracle_lib):
    model = make_model("trigram_v128")
    check_normalisation(oracle.LIB_PATH, model, np.arange(model.num_states, dtype=np.int32))


def test_normalisation_fourgram_200k_sampled(oracle_lib):
    model = make_model("fourgram_200k")
    check_normalisation(oracle.LIB_PATH, model, uniform_states(model, 3000, seed=9))


def test_normalisation_sixgram_2m_sampled(oracle_lib):
    """The 2M 6-gram with context-biasing phrases: deep phrase states and uniform ones."""
    model = make_model("sixgram_2m_phrases")
    states = np.concatenate([phrase_states(model, 4000, seed=19), uniform_states(model, 16000, seed=20)])
    check_normalisation(oracle.LIB_PATH, model, states.astype(np.int32))


def test_normalisation_tiny_with_unk(oracle_lib):
    model = tiny_model(9, 3, seed=21, n_unigrams=6)
    assert not np.isnan(model.unk_logprob)
    check_normalisation(oracle.LIB_PATH, model, np.arange(model.num_states, dtype=np.int32))


def test_unigram_model_rows_equal_unigram_row(oracle_lib):
    model = generate_model(50, [50], 1.1, seed=3)
    o = Oracle.from_model(model)
    assert o.num_states == 1
    s32, nx, _ = o.advance(np.zeros(3, np.int32))
    order, tokens, W, B = model.to_list()
    exp = np.empty(50, np.float32)
    exp[tokens[:, 0]] = W
    assert (s32 == exp).all() and (nx == 0).all()


def test_bigram_textbook_backoff(oracle_lib):
    model = generate_model(30, [30, 300], 1.0, seed=4)
    o = Oracle.from_model(model)
    order, tokens, W, B = model.to_list()
    Wd = {tuple(t[:k]): w for k, t, w in zip(order, tokens, W)}
    Bd = {tuple(t[:k]): b for k, t, b in zip(order, tokens, B)}
    s32, nx, s64 = o.advance(np.arange(o.num_states, dtype=np.int32), want64=True)
    for u in range(30):
        su = o.state_of([u])
        assert su == u + 1
        for v in range(30):
            if (u, v) in Wd:
                exp, exp_next = float(Wd[(u, v)]), v + 1
            else:
                exp, exp_next = float(Bd[(u,)]) + float(Wd[(v,)]), v + 1
            assert abs(s64[su, v] - exp) < 1e-12
            assert nx[su, v] == exp_next


def test_full_coverage_context_needs_no_backoff(oracle_lib):
    # every bigram of token 0 is listed: that context's row is its own weights
    V = 12
    model = generate_model(V, [V, 5 * V], 1.0, seed=8)
    order, tokens, W, B = model.to_list()
    full = np.array([[0, v] for v in range(V)], np.int32)
    keep = ~((order == 2) & (tokens[:, 0] == 0))
    tok2 = np.concatenate([tokens[keep], np.pad(full, ((0, 0), (0, 0)), constant_values=-1)])
    w_full = np.log(np.full(V, 1.0 / V)).astype(np.float32)
    o = Oracle(V, 2, np.concatenate([order[keep], np.full(V, 2, np.int32)]), tok2,
               np.concatenate([W[keep], w_full]), np.concatenate([B[keep], np.zeros(V, np.float32)]))
    s32, nx, _ = o.advance(np.array([o.state_of([0])], np.int32))
    assert (s32[0] == w_full).all()
    # and a context missing exactly one continuation backs off for that token only
    miss = 7
    sel = np.ones(len(o_list := tok2), bool)
    sel[len(tokens[keep]) + miss] = False
    o2 = Oracle(V, 2, np.concatenate([order[keep], np.full(V, 2, np.int32)])[sel], tok2[sel],
                np.concatenate([W[keep], w_full])[sel],
                np.concatenate([B[keep], np.zeros(V, np.float32)])[sel])
    s32b, _, _ = o2.advance(np.array([o2.state_of([0])], np.int32))
    bo = float(B[(order == 1) & (tokens[:, 0] == 0)][0])
    w1 = float(W[(order == 1) & (tokens[:, 0] == miss)][0])
    assert s32b[0, miss] == np.float32(np.float32(0.0) + np.float32(bo)) + np.float32(w1)
    assert (np.delete(s32b[0], miss) == np.delete(w_full, miss)).all()


def test_structural_invariants_fourgram_200k(oracle_lib):
    model = make_model("fourgram_200k")
    o = Oracle.from_model(model)
    states = uniform_states(model, 200, seed=12)
    _, nx, _ = o.advance(states, nthreads=8)
    N = model.max_order
    for b, s in enumerate(states):
        c = o.state_context(int(s))
        for v in range(0, model.vocab_size, 7):
            n = int(nx[b, v])
            assert n >= 0
            cn = o.state_context(n)
            assert len(cn) <= min(len(c) + 1, N - 1)
            full = c + (v,)
            assert full[len(full) - len(cn):] == cn


def test_fp32_fold_within_rounding_bound(oracle_lib):
    model = make_model("fourgram_200k")
    o = Oracle.from_model(model)
    states = uniform_states(model, 300, seed=13)
    s32, _, s64 = o.advance(states, nthreads=8, want64=True)
    # at most N-1 backoff adds plus one weight add, each rounded once (unit 2^-24)
    N = model.max_order
    bound = N * 2.0 ** -24 * (np.abs(s64) + 8.0 * N)
    assert (np.abs(s32 - s64) <= bound).all()
    assert np.abs(s32 - s64).max() < 1e-5


def test_lambda_zero_plain_is_asr_argmax(oracle_lib):
    check_lambda_zero_and_ties(oracle.LIB_PATH)


def test_ctc_rules_hand_cases(oracle_lib):
    check_ctc_rules(oracle.LIB_PATH)


def test_ctc_lambda_zero_is_textbook_greedy_ctc(oracle_lib):
    model = make_model("trigram_v128")
    o = Oracle.from_model(model)
    V = model.vocab_size
    asr = asr_logprobs((6, 80, V + 1), seed=14, blank_boost=2.0)
    # force some repeats: copy frame t-1 into frame t here and there
    asr[:, 1::5] = asr[:, 0::5][:, : asr[:, 1::5].shape[1]]
    labels, _ = o.decode(asr, MODE_CTC, 0.0)
    raw = np.argmax(asr, axis=2)
    assert (labels == raw).all()

    def collapse(row):
        out, prev = [], V
        for a in row:
            if a != V and a != prev:
                out.append(int(a))
            prev = a
        return out

    for b in range(6):
        # the advancing frames (non-blank, non-repeat) are exactly the collapsed sequence
        adv = [int(labels[b, t]) for t in range(80)
               if labels[b, t] != V and labels[b, t] != (labels[b, t - 1] if t else V)]
        assert adv == collapse(raw[b])


def test_decode_is_causal_resumable_and_the_iterated_step(oracle_lib):
    """Three invariants of a greedy decode, in every mode: frame t depends on
    frames <= t only (a ragged length cuts the labels, later frames read -1 and
    keep the state); two decodes that hand over state and last label equal one
    decode; and the decode equals the single step iterated frame by frame."""
    plain = make_model("trigram_v128")
    marked = generate_model(40, [40, 300, 400], 1.0, seed=12, bos_eos=True)
    rng = np.random.default_rng(5)
    for model, mode in ((plain, MODE_PLAIN), (plain, MODE_CTC), (plain, MODE_TRANSDUCER), (marked, MODE_AED)):
        o = Oracle.from_model(model)
        V = model.vocab_size
        B, T, cut = 7, 30, 11
        C = V if mode == MODE_PLAIN else V + 1
        asr = asr_logprobs((B, T, C), seed=int(mode) + 20, blank_boost=1.5 if mode != MODE_PLAIN else 0.0)
        starts = rng.integers(0, o.num_states, B).astype(np.int32)
        full_l, full_s = o.decode(asr, mode, 0.6, starts)
        # causal: ragged lengths
        lengths = np.array([0, 1, 5, T, 17, 29, 3], np.int32)
        l2, s2 = o.decode(asr, mode, 0.6, starts, lengths=lengths)
        for b, L in enumerate(lengths):
            assert np.array_equal(l2[b, :L], full_l[b, :L]) and (l2[b, L:] == -1).all()
            assert np.array_equal(s2[b, :L], full_s[b, :L])
            assert (s2[b, L:] == (full_s[b, L - 1] if L else starts[b])).all()
        # resumable: two decodes handing over (state, last label)
        a1, b1 = o.decode(np.ascontiguousarray(asr[:, :cut]), mode, 0.6, starts)
        prev = np.ascontiguousarray(a1[:, -1]) if mode == MODE_CTC else None
        a2, b2 = o.decode(np.ascontiguousarray(asr[:, cut:]), mode, 0.6, np.ascontiguousarray(b1[:, -1]),
                          prev=prev)
        assert np.array_equal(np.concatenate([a1, a2], 1), full_l)
        assert np.array_equal(np.concatenate([b1, b2], 1), full_s)
        # the single step iterated
        st = starts.copy()
        pv = np.full(B, V, np.int32) if mode == MODE_CTC else None
        for t in range(T):
            tok = o.greedy_step(np.ascontiguousarray(asr[:, t]), mode, 0.6, st, pv)
            assert np.array_equal(tok, full_l[:, t]) and np.array_equal(st, full_s[:, t])


def test_transducer_lambda_zero_is_raw_argmax(oracle_lib):
    """At lambda = 0 the transducer rule is the raw argmax over V + 1 classes
    (blank kept), and the state follows the emitted tokens."""
    model = make_model("trigram_v128")
    o = Oracle.from_model(model)
    V = model.vocab_size
    asr = asr_logprobs((6, 40, V + 1), seed=71, blank_boost=2.0)
    asr[0, 3, :] = -2.0                         # a full tie: index 0
    labels, states = o.decode(asr, MODE_TRANSDUCER, 0.0)
    assert np.array_equal(labels, np.argmax(asr, axis=-1))
    for b in range(asr.shape[0]):
        st = 0
        for t in range(asr.shape[1]):
            if labels[b, t] != V:
                _, nx, _ = o.advance(np.array([st], np.int32))
                st = int(nx[0, labels[b, t]])
            assert states[b, t] == st


def test_topk_reductions(oracle_lib):
    """k = 1 is the plain greedy step; lambda = 0 is a stable descending sort of the ASR row;
    k = V lists every token once, fused scores non-increasing."""
    m = make_model("trigram_v128")
    o = Oracle.from_model(m)
    V = m.vocab_size
    rng = np.random.default_rng(15)
    states = rng.integers(0, o.num_states, 40).astype(np.int32)
    asr = asr_logprobs((40, V), seed=16)
    asr[:4, :] = -2.0                                  # full ties
    tok, sc, nx = o.fused_topk(asr, 0.7, 1, states)
    st = states.copy()
    g = o.greedy_step(asr, MODE_PLAIN, 0.7, st)
    assert tok[:, 0].tolist() == g.tolist() and nx[:, 0].tolist() == st.tolist()
    tok, sc, nx = o.fused_topk(asr, 0.0, 9, states)
    order = np.argsort(-asr, axis=1, kind="stable")[:, :9]
    assert (tok == order).all()
    tok, sc, nx = o.fused_topk(asr, 1.3, V, states[:5])
    for b in range(5):
        assert sorted(tok[b].tolist()) == list(range(V))
        assert (np.diff(sc[b]) <= 0).all()
        s32, n, _ = o.advance(states[b:b + 1])
        # the fused score is lambda * lm + asr with one rounding
        assert np.abs(sc[b] - (np.float64(np.float32(1.3)) * s32[0] + asr[b])[tok[b]]).max() < 1e-5
        assert (nx[b] == n[0][tok[b]]).all()


def bos_eos_model(seed=3, V=20, counts=(20, 150, 200, 150)):
    return generate_model(V, list(counts), 1.0, seed=seed, bos_eos=True)


def test_bos_eos_normalisation_includes_final_weight(oracle_lib):
    """With </s> every context sums to one over the V tokens and </s>, so the
    final weight is pinned by the same invariant as the scores."""
    for seed in (3, 4):
        m = bos_eos_model(seed)
        o = Oracle.from_model(m)
        S = o.num_states
        states = np.arange(S, dtype=np.int32)
        s32, nx, s64 = o.advance(states, want64=True)
        fin = o.final(states).astype(np.float64)
        tot = np.exp(s64).sum(axis=1) + np.exp(fin)
        assert np.abs(tot - 1).max() < 1e-5
        assert o.start_state == m.start_state and o.state_context(o.start_state) == (m.vocab_size,)


def test_bos_eos_bruteforce_histories(oracle_lib):
    """Sentences start in <s>: every history after <s> reaches the longest listed
    context, and its token and </s> scores follow the recursion."""
    m = bos_eos_model(5, V=5, counts=(5, 18, 20, 16))
    o = Oracle.from_model(m)
    bf = BruteForce.from_model(m)
    V, eos = m.vocab_size, m.vocab_size + 1
    S = o.num_states
    s32, nx, s64 = o.advance(np.arange(S, dtype=np.int32), want64=True)
    fin = o.final(np.arange(S, dtype=np.int32))
    for L in range(0, 4):
        for w in itertools.product(range(V), repeat=L):
            h = (V,) + w
            st = o.start_state
            for t in w:
                st = int(nx[st, t])
            assert o.state_context(st) == bf.state_context(h)
            for v in range(V):
                assert abs(s64[st, v] - bf.score(h, v)) < 1e-9
            assert abs(fin[st] - bf.score(h, eos)) < 1e-5


def fmaf32(a, x, y):
    """fmaf(a, x, y) for fp32 operands, rounded once to the nearest fp32 (ties
    to even): the exact value as a fraction, then the nearer of the two fp32
    neighbours around its double rounding."""
    r = Fraction(float(a)) * Fraction(float(x)) + Fraction(float(y))
    c = np.float32(float(r))
    best = None
    for cand in (np.nextafter(c, np.float32(-np.inf)), c, np.nextafter(c, np.float32(np.inf))):
        if not np.isfinite(cand):
            continue
        d = abs(Fraction(float(cand)) - r)
        if best is None or d < best[0] or (d == best[0] and (int(cand.view(np.uint32)) & 1) == 0):
            best = (d, cand)
    return best[1]


def aed_hand_model():
    """Hand bigram model with sentence markers: tokens a = 0, b = 1, <s> = 2,
    </s> = 3.  Unigrams a (W -1, B -0.5), b (W -2, B 0), <s> (B -0.25),
    </s> (W -1.5); bigrams '<s> a' (W -0.5) and 'a </s>' (W -0.75).  Every
    weight and every sum below is a dyadic fraction, exact in fp32.
    States: 0 root, 1 'a', 2 'b', 3 '<s>' (the start state).  From state 3:
    a -> -0.5 (listed, next 1), b -> B(<s>) + W(b) = -2.25 (next 2), final
    weight B(<s>) + W(</s>) = -1.75.  From state 1: a -> B(a) + W(a) = -1.5
    (next 1), b -> -2.5 (next 2), final weight -0.75 (listed 'a </s>')."""
    rows = [((0,), -1.0, -0.5), ((1,), -2.0, 0.0), ((2,), -1.0, -0.25), ((3,), -1.5, 0.0),
            ((2, 0), -0.5, 0.0), ((0, 3), -0.75, 0.0)]
    order = np.array([len(r[0]) for r in rows], np.int32)
    tokens = np.full((len(rows), 2), -1, np.int32)
    for i, r in enumerate(rows):
        tokens[i, :len(r[0])] = r[0]
    W = np.array([r[1] for r in rows], np.float32)
    B = np.array([r[2] for r in rows], np.float32)
    return (2, 2, order, tokens, W, B)


def check_aed_ties(lib_path):
    """AED (Section 2.3): <eos> is class V, after every token, so an exact tie
    between a token and <eos> goes to the token (lowest index); <eos> wins only
    when strictly larger, and then the state stays."""
    o = Oracle(*aed_hand_model(), lib_path=lib_path, bos_eos=True)
    assert o.start_state == 3 and o.state_context(3) == (2,)
    s32, nx, _ = o.advance(np.array([3, 1], np.int32))
    assert s32.tolist() == [[-0.5, -2.25], [-1.5, -2.5]] and nx.tolist() == [[1, 2], [1, 2]]
    assert o.final(np.array([3, 1], np.int32)).tolist() == [-1.75, -0.75]
    cases = [
        # (state, lambda, asr [a, b, <eos>], label, state after)
        (3, 0.0, [-3.0, -1.0, -1.0], 1, 2),      # raw tie b = <eos>: b
        (3, 0.0, [-1.0, -1.0, -1.0], 0, 1),      # three-way tie: a
        (3, 0.0, [-3.0, -1.0, -0.5], 2, 3),      # <eos> strictly larger: ends, state kept
        (3, 0.5, [-5.0, -0.5, -0.75], 1, 2),     # fused: b = -1.125 - 0.5, <eos> = -0.875 - 0.75, tie
        (3, 0.5, [-5.0, -0.5, -0.5], 2, 3),      # <eos> -1.375 above b -1.625
        (1, 0.5, [-1.0, -3.0, -1.375], 0, 1),    # a = -0.75 - 1, <eos> = -0.375 - 1.375, tie
        (1, 0.5, [-1.0, -3.0, -1.25], 2, 1),     # <eos> -1.625 above a -1.75
    ]
    for s0, lam, row, lab, s1 in cases:
        st = np.array([s0], np.int32)
        tok = o.greedy_step(np.array([row], np.float32), MODE_AED, lam, st)
        assert (int(tok[0]), int(st[0])) == (lab, s1), (s0, lam, row)


def test_aed_hand_ties(oracle_lib):
    check_aed_ties(oracle.LIB_PATH)


def test_aed_mode_rules(oracle_lib):
    """lambda = 0: the raw argmax over V tokens and <eos> (class V); <eos> keeps
    the state; otherwise the state follows the token."""
    m = bos_eos_model(6)
    o = Oracle.from_model(m)
    V = m.vocab_size
    rng = np.random.default_rng(17)
    states = rng.integers(0, o.num_states, 60).astype(np.int32)
    asr = asr_logprobs((60, V + 1), seed=18)
    asr[:10, V] = 1.0                            # <eos> wins for ten rows
    st = states.copy()
    tok = o.greedy_step(asr, MODE_AED, 0.0, st)
    assert tok.tolist() == np.argmax(asr, axis=1).tolist()
    _, nx, _ = o.advance(states)
    for b in range(60):
        exp = states[b] if tok[b] == V else nx[b, tok[b]]
        assert st[b] == exp
    # lambda > 0: <eos> is scored with the final weight
    st = states.copy()
    tok = o.greedy_step(asr, MODE_AED, 0.8, st)
    s32, _, _ = o.advance(states)
    fin = o.final(states)
    lam = np.float32(0.8)
    for b in range(60):
        f = [fmaf32(lam, s32[b, v], asr[b, v]) for v in range(V)] + [fmaf32(lam, fin[b], asr[b, V])]
        assert tok[b] == int(np.argmax(np.array(f, np.float32)))   # first maximal index


def test_repair_of_pruned_lists(oracle_lib):
    check_repair(oracle.LIB_PATH)


def test_generator_and_oracle_number_states_alike(oracle_lib):
    check_generator_ids(oracle.LIB_PATH)


def test_error_codes():
    fx, (V, N, order, tokens, W, B) = fig1_list()
    with pytest.raises(oracle.OracleError) as e:
        Oracle(V, N, np.append(order, 1), np.vstack([tokens, tokens[:1]]), np.append(W, 0), np.append(B, 0))
    assert e.value.code == -4
    bad = tokens.copy(); bad[3, 0] = V
    with pytest.raises(oracle.OracleError) as e:
        Oracle(V, N, order, bad, W, B)
    assert e.value.code == -2
    with pytest.raises(oracle.OracleError) as e:
        Oracle(V, N, order[1:], tokens[1:], W[1:], B[1:])          # 'the' unigram missing, no <unk>
    assert e.value.code == -7


# ------------------------------------------------- planted mistakes are caught

MUTANTS = {
    "dropped backoff term": ("float b = rc >= 0 ? m->B[rc] : 0.0f;", "float b = 0.0f; (void)rc;"),
    "backoff sign": ("float b = rc >= 0 ? m->B[rc] : 0.0f;", "float b = rc >= 0 ? -m->B[rc] : 0.0f;"),
    "backoff of the prefix": ("int64_t rc = lookup(m, c + (n - k), k);", "int64_t rc = lookup(m, c, k);"),
    "context prefix instead of suffix": ("memcpy(g, c + (n - k), sizeof(int32_t) * (size_t)k);",
                                         "memcpy(g, c, sizeof(int32_t) * (size_t)k);"),
    "next drops the token": ("*next = (int32_t)longest_state_suffix(m, g, k + 1);",
                             "*next = (int32_t)longest_state_suffix(m, g, k);"),
    "reversed numbering": ("if (ta[i] != tb[i]) return ta[i] < tb[i] ? -1 : 1;",
                           "if (ta[i] != tb[i]) return ta[i] > tb[i] ? -1 : 1;"),
    "transposed fusion operands": ("float f = fmaf(lambda, lm[v], asr[v]);", "float f = fmaf(lambda, asr[v], lm[v]);"),
    "repeat rescored": ("if (a == V || (mode == MODE_CTC && a == *prev)) {", "if (a == V) {"),
    "last index wins ties": ("if (best < 0 || f > bestval) { best = v; bestval = f; }",
                             "if (best < 0 || f >= bestval) { best = v; bestval = f; }"),
    "<eos> wins ties": ("if (f > bestval) return V;", "if (f >= bestval) return V;"),
    "repair weighs an added n-gram with itself": ("if (!l->added[r] || l->ord[r] < kmax)", "if (1)"),
    "repair adds no suffixes": ("if (!(special && t[k - 1] == V + 1))\n", "if (0)\n"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = open(oracle.SRC_PATH).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for '{name}' not found exactly once"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib = str(tmp_path / "libmutant.so")
    subprocess.run(["gcc", *oracle.CFLAGS, "-w", "-o", lib, str(path), "-lm"], check=True)
    small = make_model("trigram_v128")
    checks = [
        lambda: check_worked_example(lib),
        lambda: check_bruteforce_tiny(lib, seeds=(0, 1, 2)),
        lambda: check_normalisation(lib, small, np.arange(small.num_states, dtype=np.int32)),
        lambda: check_lambda_zero_and_ties(lib),
        lambda: check_ctc_rules(lib),
        lambda: check_generator_ids(lib),
        lambda: check_repair(lib, seeds=(6,)),
        lambda: check_aed_ties(lib),
    ]
    caught = 0
    for chk in checks:
        try:
            chk()
        except (AssertionError, oracle.OracleError):
            caught += 1
    assert caught >= 1, f"no pin caught the planted mistake '{name}'"
