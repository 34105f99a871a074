"""The seeded generators: closure, counts, determinism and the normalising construction."""

import numpy as np

from synth import (WORKLOADS, asr_logprobs, generate_model, lookup_ids, make_model,
                   phrase_states, state_ids_of, tiny_model, uniform_states)


def _closure_ok(model):
    for k in range(2, model.max_order + 1):
        t = model.level_tokens(k)
        assert (lookup_ids(model, t[:, :-1]) >= 0).all(), f"prefix closure at order {k}"
        assert (lookup_ids(model, t[:, 1:]) >= 0).all(), f"suffix closure at order {k}"
        # lexicographic order, no duplicates
        key = np.lexsort(t.T[::-1])
        assert (key == np.arange(len(t))).all()
        assert (np.diff(model.levels[k].pid * model.vocab_size + model.levels[k].tok) > 0).all()


def _construction_identity(model, tol=1e-6):
    """Stored mass Z(c) = sum_E P(v|c) + exp(B(c)) * (Z(c[1:]) - sum_E P(v|c[1:])) is 1 for every context."""
    V = model.vocab_size
    z1 = np.exp(model.levels[1].W.astype(np.float64)).sum()
    if not np.isnan(model.unk_logprob):
        z1 += (V - len(model.levels[1].tok)) * np.exp(np.float64(model.unk_logprob))
    assert abs(z1 - 1.0) < 1e-6
    z = [np.array([z1])]
    for k in range(2, model.max_order + 1):
        lv, prev = model.levels[k], model.levels[k - 1]
        n = len(prev.tok)
        m = np.bincount(lv.pid, weights=np.exp(lv.W.astype(np.float64)), minlength=n)
        l = np.bincount(lv.pid, weights=np.exp(prev.W[lv.sid].astype(np.float64)), minlength=n)
        zlow = z[-1][prev.sid]
        tot = m + np.exp(prev.B.astype(np.float64)) * (zlow - l)
        tot[np.bincount(lv.pid, minlength=n) == V] = m[np.bincount(lv.pid, minlength=n) == V]
        assert np.abs(tot - 1.0).max() < tol, (k, np.abs(tot - 1.0).max())
        z.append(tot)


def test_workload_counts_and_closure():
    for key in ("trigram_v128", "fourgram_200k"):
        spec = WORKLOADS[key]
        m = make_model(key)
        assert m.counts == list(spec.counts)
        assert m.num_states == 1 + sum(spec.counts[:-1])
        _closure_ok(m)
        _construction_identity(m)


def test_tiny_models_closed_and_normalised():
    for seed in range(5):
        m = tiny_model(5 + seed, 2 + seed % 4, seed=seed)
        _closure_ok(m)
        _construction_identity(m)
    m = tiny_model(9, 3, seed=21, n_unigrams=6)
    _closure_ok(m)
    _construction_identity(m)


def test_bos_eos_models_closed_and_normalised():
    for seed in range(3):
        m = generate_model(16, [16, 120, 150, 100], 1.0, seed=seed, bos_eos=True)
        V = m.vocab_size
        o, t, W, B = m.to_list()
        for i in range(len(o)):
            row = t[i, :o[i]].tolist()
            assert V not in row[1:] and (V + 1) not in row[:-1]
        # every context sums to one over the V tokens and </s> (construction identity)
        z1 = np.exp(m.levels[1].W.astype(np.float64))[m.levels[1].tok != V].sum()
        assert abs(z1 - 1) < 1e-6
        for k in range(2, m.max_order + 1):
            lv = m.levels[k]
            assert (m.levels[k - 1].tok[lv.pid] != V + 1).all()     # </s> is never extended
            assert (lv.tok != V).all()                             # <s> is never predicted
        assert m.start_state == state_ids_of(m, np.array([[V]]))[0]


def test_deterministic_from_seed():
    a = generate_model(64, [64, 500, 400], 1.1, seed=5).to_list()
    b = generate_model(64, [64, 500, 400], 1.1, seed=5).to_list()
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_shuffled_list_is_a_permutation():
    m = make_model("trigram_v128")
    o1, t1, w1, b1 = m.to_list()
    o2, t2, w2, b2 = m.to_list(shuffle_seed=1)
    k1 = np.lexsort(np.column_stack([t1, o1]).T[::-1])
    k2 = np.lexsort(np.column_stack([t2, o2]).T[::-1])
    assert np.array_equal(t1[k1], t2[k2]) and np.array_equal(w1[k1], w2[k2])


def test_phrase_model_and_deep_states():
    # a scaled-down version of the context-biasing recipe
    phrases = [np.array(p) for p in ([1, 2, 3, 4, 5, 6], [7, 8, 9, 10, 11], [3, 4, 5, 6, 7, 8, 9])]
    m = generate_model(32, [32, 200, 300, 200, 100, 30], 1.05, seed=2, phrases=phrases)
    _closure_ok(m)
    _construction_identity(m)
    st = phrase_states(m, 16, seed=1)
    first5 = m.state_offset(5)
    assert (st >= first5).all() and (st < m.num_states).all()


def test_uniform_states_and_asr():
    m = make_model("trigram_v128")
    s = uniform_states(m, 1000, seed=3)
    assert s.dtype == np.int32 and s.min() >= 0 and s.max() < m.num_states
    a = asr_logprobs((3, 7, 129), seed=1, blank_boost=4.0)
    assert a.dtype == np.float32 and a.shape == (3, 7, 129)
    assert np.abs(np.exp(a.astype(np.float64)).sum(-1) - 1).max() < 1e-5
    assert (np.argmax(a, -1) == 128).mean() > 0.0
