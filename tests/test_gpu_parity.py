"""GPU parity of the HIP kernels with the CPU oracle, through the C ABI.

Next states and labels must match bit for bit; scores within 1e-5 nats (the
kernels take the same fp32 fold as the oracle's fp32 result, so they are
expected to be bit-exact and the test reports any difference).  Every case
prints its name before it touches the GPU.
"""

import os
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

import paper_2505_22857_amd as ng  # noqa: E402
from oracle import MODE_AED, MODE_CTC, MODE_PLAIN, MODE_TRANSDUCER, Oracle  # noqa: E402
from synth import (WORKLOADS, asr_logprobs, generate_model, make_model, phrase_states,  # noqa: E402
                   seed_for, tiny_model, uniform_states)

TOL = 1e-5
NTHREADS = max(1, min(16, len(os.sched_getaffinity(0))))


def case(msg):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="session")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch.device("cuda:0")


_PAIRS = {}


def pair(key, make):
    """(model, uploaded library trie, oracle), built once per session."""
    if key not in _PAIRS:
        m = make()
        lm = ng.NgpuLM.from_model(m, shuffle_seed=17).upload("cuda:0")
        o = Oracle.from_model(m)
        _PAIRS[key] = (m, lm, o)
    return _PAIRS[key]


def model_pair(key):
    return pair(key, lambda: make_model(key))


def run_advance(lm, states_np, dev):
    st = torch.from_numpy(np.ascontiguousarray(states_np, np.int32)).to(dev)
    sc, nx = lm.advance(st)
    torch.cuda.synchronize()
    return sc.cpu().numpy(), nx.cpu().numpy()


def assert_rows(name, sc, nx, o_s32, o_nx):
    assert np.array_equal(nx, o_nx), f"{name}: next states differ at {np.argwhere(nx != o_nx)[:5]}"
    d = np.abs(sc.astype(np.float64) - o_s32)
    assert np.isfinite(sc).all()
    assert d.max() <= TOL, f"{name}: max |score diff| {d.max()}"
    inexact = int((sc != o_s32).sum())
    print(f"  {name}: {sc.shape[0]} rows, max |diff| {d.max():.3g}, non-bit-exact {inexact}", flush=True)


def check_advance(name, m, lm, o, states, dev, rows=None):
    case(f"advance {name} B={len(states)}")
    sc, nx = run_advance(lm, states, dev)
    assert lm.check_states() == 0
    idx = np.arange(len(states)) if rows is None else rows
    o_s32, o_nx, _ = o.advance(states[idx], nthreads=NTHREADS)
    assert_rows(name, sc[idx], nx[idx], o_s32, o_nx)
    return sc, nx


# ------------------------------------------------------------------ advance

def test_advance_trigram_every_state(dev):
    m, lm, o = model_pair("trigram_v128")
    check_advance("trigram V=128 all states", m, lm, o, np.arange(m.num_states, dtype=np.int32), dev)


@pytest.mark.parametrize("B", [1, 33, 1024, 1025, 32 * 64])
def test_advance_4gram_200k(dev, B):
    m, lm, o = model_pair("fourgram_200k")
    check_advance("4-gram 200k", m, lm, o, uniform_states(m, B, seed=seed_for("fourgram_200k") + B), dev)


def test_advance_6gram_2m_deep_phrase_states(dev):
    m, lm, o = model_pair("sixgram_2m_phrases")
    st = phrase_states(m, WORKLOADS["sixgram_2m_phrases"].batch, seed=seed_for("sixgram_2m_phrases"))
    check_advance("6-gram 2M phrase states", m, lm, o, st, dev)
    check_advance("6-gram 2M uniform", m, lm, o, uniform_states(m, 1000, seed=seed_for("sixgram_2m_phrases") + 1), dev)


def test_advance_6gram_2m_rows_normalised(dev):
    """Every row of 10^5 sampled states sums to one (a property of the generated
    model), on the GPU's scores."""
    m, lm, o = model_pair("sixgram_2m_phrases")
    st = np.concatenate([phrase_states(m, 20000, seed=seed_for("sixgram_2m_phrases") + 2),
                         uniform_states(m, 80000, seed=seed_for("sixgram_2m_phrases") + 3)]).astype(np.int32)
    case(f"advance 6-gram 2M normalisation B={len(st)}")
    sc, nx = lm.advance(torch.from_numpy(st).to(dev))
    torch.cuda.synchronize()
    assert lm.check_states() == 0
    tot = torch.exp(sc.double()).sum(dim=1)
    err = float((tot - 1).abs().max())
    print(f"  6-gram 2M max |sum - 1| over {len(st)} rows: {err:.3g}", flush=True)
    assert err < 1e-5
    assert int(nx.min()) >= 0 and int(nx.max()) < m.num_states


def test_advance_6gram_20m_64_batches_of_512(dev):
    """64 independent 512-hypothesis calls, every row against the oracle."""
    m, lm, o = model_pair("sixgram_20m")
    R, Bb = 64, 512
    states = np.concatenate([uniform_states(m, Bb, seed=seed_for("sixgram_20m") + r) for r in range(R)])
    st = torch.from_numpy(states).to(dev)
    sc = torch.empty((R * Bb, m.vocab_size), dtype=torch.float32, device=dev)
    nx = torch.empty((R * Bb, m.vocab_size), dtype=torch.int32, device=dev)
    case(f"advance 6-gram 20M {R} calls of B={Bb}")
    for r in range(R):
        sl = slice(r * Bb, (r + 1) * Bb)
        lm.advance(st[sl], sc[sl], nx[sl])
    torch.cuda.synchronize()
    assert lm.check_states() == 0
    o_s32, o_nx, _ = o.advance(states, nthreads=NTHREADS)
    assert_rows(f"6-gram 20M {R} x {Bb}", sc.cpu().numpy(), nx.cpu().numpy(), o_s32, o_nx)


def test_advance_6gram_20m_bench_launch_sampled(dev):
    """The benchmark's launch (128 batches of 512 in one call): sampled rows vs the
    oracle, and per-row normalisation (a property of the generated model) on every row."""
    m, lm, o = model_pair("sixgram_20m")
    B = 128 * 512
    states = uniform_states(m, B, seed=seed_for("sixgram_20m") + 1000)
    case(f"advance 6-gram 20M B={B}")
    st = torch.from_numpy(states).to(dev)
    sc, nx = lm.advance(st)
    torch.cuda.synchronize()
    assert lm.check_states() == 0
    rows = np.random.default_rng(3).choice(B, 2048, replace=False)
    rows = np.concatenate([rows, [0, B - 1]])
    o_s32, o_nx, _ = o.advance(states[rows], nthreads=NTHREADS)
    rt = torch.from_numpy(rows).to(dev)
    assert_rows("6-gram 20M B=65536 sampled", sc[rt].cpu().numpy(), nx[rt].cpu().numpy(), o_s32, o_nx)
    tot = torch.exp(sc.double()).sum(dim=1)
    assert float((tot - 1).abs().max()) < 1e-5
    assert int(nx.min()) >= 0 and int(nx.max()) < m.num_states


@pytest.mark.parametrize("which", ["4gram_200k", "V800", "V1025", "N10"])
def test_advance_grouped_mapping_with_bad_states(dev, which):
    """Batches of 20480 and more take the XCD-grouped mapping: every row, including
    rows of out-of-range states (written by exactly one owner), vs the oracle.
    V in (768, 1024] runs it with two wavefronts per hypothesis, one per
    512-token half (V = 800: a ragged second half); V = 1025 with one.
    N10: a 10-gram, whose order-9 states have chain records longer than the
    scan preloads."""
    if which == "4gram_200k":
        m, lm, o = model_pair("fourgram_200k")
        B = 40000
    elif which == "V800":
        m, lm, o = pair("V800N4", lambda: generate_model(800, [800, 4800, 4800, 4800], 1.0, seed=804))
        B = 20488
    elif which == "V1025":
        m, lm, o = pair("V1025N4", lambda: generate_model(1025, [1025, 6150, 6150, 6150], 1.0, seed=1029))
        B = 20481
    else:
        m, lm, o = pair("V16N10", lambda: generate_model(16, [16, 120, 200, 200, 180, 160, 140, 120, 100, 80],
                                                          1.0, seed=26))
        B = 32800
    states = uniform_states(m, B, seed=23)
    bad = np.random.default_rng(24).choice(B, 37, replace=False)
    states[bad[:20]] = -5
    states[bad[20:]] = m.num_states + np.arange(17)
    case(f"advance grouped {which} B={B} with {len(bad)} bad states")
    sc, nx = run_advance(lm, states, dev)
    assert lm.check_states() == len(bad)
    good = np.setdiff1d(np.arange(B), bad)
    assert np.isnan(sc[bad]).all() and (nx[bad] == -1).all()
    o_s32, o_nx, _ = o.advance(states[good], nthreads=NTHREADS)
    assert_rows(f"grouped {which}", sc[good], nx[good], o_s32, o_nx)


@pytest.mark.parametrize("V,N", [(5, 3), (1000, 3), (1025, 4), (4096, 3), (16, 10)])
def test_advance_odd_shapes(dev, V, N):
    if N == 10:
        counts = [V, 120, 200, 200, 180, 160, 140, 120, 100, 80]
    else:
        counts = [V, min(V * V // 2, 6 * V)] + [min(V * V // 2, 6 * V)] * (N - 2)
    m, lm, o = pair(f"V{V}N{N}", lambda: generate_model(V, counts, 1.0, seed=V + N))
    st = np.arange(m.num_states, dtype=np.int32)
    if len(st) > 3000:
        st = uniform_states(m, 3001, seed=1)
    check_advance(f"V={V} N={N}", m, lm, o, st, dev)


@pytest.mark.parametrize("V,N", [(5, 3), (300, 3), (700, 3), (1025, 4), (4096, 3), (16, 10)])
def test_advance_small_batches_every_stripe_count(dev, V, N):
    """Batches of up to 1024 hypotheses run with one wavefront per 256-token
    stripe, at most four: V = 5 and 16 one stripe, 300 two, 700 three stripes
    on two wavefronts, 1025 (no 16-byte stores) and 4096 four.  Out-of-range
    states among them give rows of NaN / -1 and are counted."""
    if N == 10:
        counts = [V, 120, 200, 200, 180, 160, 140, 120, 100, 80]
    else:
        counts = [V, min(V * V // 2, 6 * V)] + [min(V * V // 2, 6 * V)] * (N - 2)
    m, lm, o = pair(f"V{V}N{N}", lambda: generate_model(V, counts, 1.0, seed=V + N))
    st = uniform_states(m, 700, seed=V + 2)
    st[[3, 400]] = [-1, m.num_states]
    case(f"advance small batch V={V} N={N} B={len(st)} with 2 bad states")
    sc, nx = run_advance(lm, st, dev)
    assert lm.check_states() == 2
    assert np.isnan(sc[[3, 400]]).all() and (nx[[3, 400]] == -1).all()
    good = np.setdiff1d(np.arange(len(st)), [3, 400])
    o_s32, o_nx, _ = o.advance(st[good], nthreads=NTHREADS)
    assert_rows(f"V={V} N={N} small batch", sc[good], nx[good], o_s32, o_nx)


def ten_gram_pair():
    return pair("V1024N10", lambda: generate_model(
        1024, [1024, 20000, 40000, 40000, 30000, 20000, 15000, 10000, 8000, 6000], 1.0, seed=1010))


def test_ten_gram_vocab_1024(dev):
    """A 10-gram over V = 1024, the order and vocabulary of the paper's LMs:
    chains of up to nine records, in the plain and the XCD-grouped mapping,
    and the decode launch."""
    m, lm, o = ten_gram_pair()
    small = uniform_states(m, 3000, seed=101)
    check_advance("10-gram plain mapping", m, lm, o, small, dev)
    big = uniform_states(m, 40000, seed=102)
    rows = np.random.default_rng(103).choice(len(big), 3000, replace=False)
    check_advance("10-gram grouped mapping", m, lm, o, big, dev, rows=rows)
    Bq, T = 64, 60
    asr = asr_logprobs((Bq, T, 1025), seed=104, blank_boost=1.0)
    starts = uniform_states(m, Bq, seed=105)
    for mode in (MODE_PLAIN, MODE_CTC):
        a = asr if mode == MODE_CTC else np.ascontiguousarray(asr[:, :, :1024])
        case(f"10-gram decode launch mode={mode}")
        gl, gs, _, _ = gpu_decode_launch(lm, a, mode, 0.5, starts, dev)
        ol, os_ = o.decode(a, mode, 0.5, starts, nthreads=NTHREADS)
        assert np.array_equal(gl, ol) and np.array_equal(gs, os_)


def test_repaired_pruned_model(dev):
    """A pruned (not closed) 4-gram built with closure repair: advance and the
    decode launch against the oracle on the oracle's own repair of the list."""
    from oracle import repair_list
    from synth import pruned_list
    m0 = make_model("fourgram_200k")
    o, t, W, B = pruned_list(m0, 0.2, seed=11)
    V, N = m0.vocab_size, m0.max_order
    lm = ng.NgpuLM(V, N, o, t, W, B, m0.unk_logprob, repair=True).upload(dev)
    R = repair_list(V, N, o, t, W, B, m0.unk_logprob)
    orc = Oracle(V, N, *R, m0.unk_logprob)
    assert lm.num_states == orc.num_states
    states = np.concatenate([np.arange(0, lm.num_states, 37), [lm.num_states - 1]]).astype(np.int32)
    check_advance("repaired pruned 4-gram 200k", None, lm, orc, states, dev)
    Bq, T = 48, 40
    starts = np.random.default_rng(13).integers(0, lm.num_states, Bq).astype(np.int32)
    asr = asr_logprobs((Bq, T, V + 1), seed=14, blank_boost=1.0)
    for mode in (MODE_PLAIN, MODE_CTC):
        a = asr if mode == MODE_CTC else np.ascontiguousarray(asr[:, :, :V])
        case(f"repaired pruned 4-gram 200k decode launch mode={mode}")
        gl, gs, _, _ = gpu_decode_launch(lm, a, mode, 0.5, starts, dev)
        ol, os_ = orc.decode(a, mode, 0.5, starts, nthreads=NTHREADS)
        assert np.array_equal(gl, ol) and np.array_equal(gs, os_)


def test_advance_unigram_and_unk_models(dev):
    m, lm, o = pair("n1", lambda: generate_model(77, [77], 1.0, seed=2))
    check_advance("N=1", m, lm, o, np.zeros(5, np.int32), dev)
    m, lm, o = pair("unk", lambda: tiny_model(9, 3, seed=21, n_unigrams=6))
    check_advance("unk", m, lm, o, np.arange(m.num_states, dtype=np.int32), dev)


def test_advance_empty_and_out_of_range(dev):
    m, lm, o = model_pair("trigram_v128")
    case("advance B=0")
    sc, nx = lm.advance(torch.zeros(0, dtype=torch.int32, device=dev))
    assert sc.shape == (0, m.vocab_size)
    case("advance with out-of-range states")
    st = np.array([0, -1, m.num_states, 5], np.int32)
    sc, nx = run_advance(lm, st, dev)
    assert lm.check_states() == 2
    assert lm.check_states() == 0          # the count clears
    assert np.isnan(sc[1]).all() and (nx[1] == -1).all() and (nx[2] == -1).all()
    o_s32, o_nx, _ = o.advance(st[[0, 3]])
    assert_rows("valid rows next to bad ones", sc[[0, 3]], nx[[0, 3]], o_s32, o_nx)


# ------------------------------------------------------------------ fused step

def gpu_decode(lm, asr_np, mode, lam, starts, dev):
    """Frame loop over fused_greedy_step; returns labels and states after each frame."""
    B, T, C = asr_np.shape
    asr = torch.from_numpy(asr_np).to(dev)
    st = torch.from_numpy(np.ascontiguousarray(starts, np.int32)).to(dev)
    prev = torch.full((B,), lm.vocab_size, dtype=torch.int32, device=dev)
    labels = torch.empty((B, T), dtype=torch.int32, device=dev)
    states = torch.empty((B, T), dtype=torch.int32, device=dev)
    tok = torch.empty(B, dtype=torch.int32, device=dev)
    for t in range(T):
        lm.fused_greedy_step(asr[:, t, :], lam, st, prev if mode == MODE_CTC else None, mode=mode, tokens=tok)
        labels[:, t] = tok
        states[:, t] = st
    torch.cuda.synchronize()
    return labels.cpu().numpy(), states.cpu().numpy()


def check_decode(name, lm, o, asr, mode, lam, starts, dev):
    case(f"fused {name} B={asr.shape[0]} T={asr.shape[1]}")
    gl, gs = gpu_decode(lm, asr, mode, lam, starts, dev)
    assert lm.check_states() == 0
    ol, os_ = o.decode(asr, mode, lam, starts, nthreads=NTHREADS)
    bad = np.argwhere(gl != ol)
    assert len(bad) == 0, f"{name}: labels differ first at (b, t) = {bad[0]}"
    assert np.array_equal(gs, os_), f"{name}: states differ"
    print(f"  {name}: {gl.size} decisions identical", flush=True)
    return gl, gs


def test_fused_plain_trigram(dev):
    m, lm, o = model_pair("trigram_v128")
    spec = WORKLOADS["trigram_v128"]
    asr = asr_logprobs((spec.batch, spec.steps, m.vocab_size), seed=seed_for("trigram_v128") + 50)
    check_decode("plain trigram V=128", lm, o, asr, MODE_PLAIN, spec.lam, np.zeros(spec.batch, np.int32), dev)


def test_fused_plain_4gram_200k_with_advance_every_step(dev):
    m, lm, o = model_pair("fourgram_200k")
    spec = WORKLOADS["fourgram_200k"]
    starts = uniform_states(m, spec.batch, seed=seed_for("fourgram_200k") + 77)
    asr = asr_logprobs((spec.batch, spec.steps, m.vocab_size), seed=seed_for("fourgram_200k") + 50)
    gl, gs = check_decode("plain 4-gram 200k", lm, o, asr, MODE_PLAIN, spec.lam, starts, dev)
    # the advance query at every step's states
    visited = np.concatenate([starts, gs[:, :-1].reshape(-1)]).astype(np.int32)
    check_advance("4-gram 200k states along the decode", m, lm, o, visited, dev)


_CTC = {}


def ctc_data():
    """The 256 x 1000 CTC workload: the ASR tensor and the oracle's decode of it, computed once."""
    if not _CTC:
        m, lm, o = model_pair("sixgram_20m")
        spec = WORKLOADS["ctc_b256_t1000"]
        V = m.vocab_size
        asr = asr_logprobs((spec.batch, spec.steps, V + 1), seed=seed_for("ctc_b256_t1000"), blank_boost=spec.blank_boost)
        _CTC["asr"] = asr
        _CTC["oracle"] = o.decode(asr, MODE_CTC, spec.lam, np.zeros(spec.batch, np.int32), nthreads=NTHREADS)
    return _CTC["asr"], _CTC["oracle"]


def test_fused_ctc_256x1000_per_frame(dev):
    m, lm, o = model_pair("sixgram_20m")
    spec = WORKLOADS["ctc_b256_t1000"]
    V = m.vocab_size
    asr, (ol, os_) = ctc_data()
    case(f"fused CTC per-frame steps, 20M 6-gram, B={spec.batch} T={spec.steps}")
    gl, gs = gpu_decode(lm, asr, MODE_CTC, spec.lam, np.zeros(spec.batch, np.int32), dev)
    assert lm.check_states() == 0
    assert np.array_equal(gl, ol) and np.array_equal(gs, os_)
    print(f"  CTC 256x1000 per-frame: {gl.size} decisions identical, blank labels {(gl == V).mean():.3f}", flush=True)


# ------------------------------------------------------------------ whole decode in one launch

def gpu_decode_launch(lm, asr_np, mode, lam, starts, dev, lengths=None, prev0=None):
    B, T, C = asr_np.shape
    asr = torch.from_numpy(asr_np).to(dev)
    st = torch.from_numpy(np.ascontiguousarray(starts, np.int32)).to(dev)
    prev = None
    if mode == MODE_CTC:
        p0 = np.full(B, lm.vocab_size, np.int32) if prev0 is None else prev0
        prev = torch.from_numpy(np.ascontiguousarray(p0, np.int32)).to(dev)
    ln = torch.from_numpy(np.ascontiguousarray(lengths, np.int32)).to(dev) if lengths is not None else None
    lst = torch.full((B, T), -9, dtype=torch.int32, device=dev)
    lab = lm.fused_greedy_decode(asr, lam, st, prev, lengths=ln, mode=mode, label_states=lst)
    torch.cuda.synchronize()
    return (lab.cpu().numpy(), lst.cpu().numpy(), st.cpu().numpy(),
            prev.cpu().numpy() if prev is not None else None)


def test_decode_launch_ctc_256x1000(dev):
    m, lm, o = model_pair("sixgram_20m")
    spec = WORKLOADS["ctc_b256_t1000"]
    asr, (ol, os_) = ctc_data()
    case(f"decode launch CTC, 20M 6-gram, B={spec.batch} T={spec.steps}")
    gl, gs, fin, fprev = gpu_decode_launch(lm, asr, MODE_CTC, spec.lam, np.zeros(spec.batch, np.int32), dev)
    assert lm.check_states() == 0
    bad = np.argwhere(gl != ol)
    assert len(bad) == 0, f"labels differ first at {bad[0]}"
    assert np.array_equal(gs, os_)
    assert np.array_equal(fin, os_[:, -1]) and np.array_equal(fprev, ol[:, -1])
    print(f"  CTC 256x1000 one launch: {gl.size} decisions identical", flush=True)


def test_decode_launch_20m_register_rows(dev):
    """The 20M 6-gram decoded with one wavefront per utterance and the ASR and
    4-byte dense rows in registers (4096 utterances x 24 frames, the shape of
    the benchmark's large decode), from uniformly drawn states (deep chains)
    and from the empty context, against the oracle."""
    m, lm, o = model_pair("sixgram_20m")
    V, B, T = m.vocab_size, 4096, 24
    asr = asr_logprobs((B, T, V + 1), seed=91, blank_boost=4.0)
    starts = uniform_states(m, B, seed=92)
    starts[::2] = 0
    for mode in (MODE_CTC, MODE_PLAIN):
        a = asr if mode != MODE_PLAIN else np.ascontiguousarray(asr[:, :, :V])
        case(f"decode launch 20M register rows B={B} T={T} mode={mode}")
        gl, gs, _, _ = gpu_decode_launch(lm, a, mode, 0.5, starts, dev)
        assert lm.check_states() == 0
        ol, os_ = o.decode(a, mode, 0.5, starts, nthreads=NTHREADS)
        bad = np.argwhere(gl != ol)
        assert len(bad) == 0, f"labels differ first at {bad[0]}"
        assert np.array_equal(gs, os_)


@pytest.mark.parametrize("mode", [MODE_PLAIN, MODE_CTC, MODE_TRANSDUCER])
def test_decode_launch_modes_ragged_lengths(dev, mode):
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    B, T = 37, 90
    starts = uniform_states(m, B, seed=31)
    C = V if mode == MODE_PLAIN else V + 1
    asr = asr_logprobs((B, T, C), seed=32, blank_boost=2.0 if mode != MODE_PLAIN else 0.0)
    lengths = np.random.default_rng(33).integers(0, T + 1, B).astype(np.int32)
    lengths[:3] = [0, T, 1]
    case(f"decode launch mode={mode} B={B} T={T} ragged")
    gl, gs, fin, fprev = gpu_decode_launch(lm, asr, mode, 0.6, starts, dev, lengths=lengths)
    assert lm.check_states() == 0
    ol, os_ = o.decode(asr, mode, 0.6, starts, nthreads=NTHREADS, lengths=lengths)
    assert np.array_equal(gl, ol)
    assert np.array_equal(gs, os_)
    assert np.array_equal(fin, os_[:, -1])


@pytest.mark.parametrize("B", [513, 1100, 5000])
def test_fused_larger_batches(dev, B):
    """Batches above 512 hypotheses: the whole decode runs with one wavefront
    per hypothesis instead of four (the per-frame step from 1025 on, so 513
    covers its four-wavefront path at that size), with the ASR rows and the
    4-byte dense rows in registers (this model has them)."""
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    T = 16
    starts = uniform_states(m, B, seed=B)
    asr = asr_logprobs((B, T, V + 1), seed=B + 1, blank_boost=1.0)
    lengths = np.random.default_rng(B + 2).integers(0, T + 1, B).astype(np.int32)
    for mode in (MODE_PLAIN, MODE_CTC):
        a = asr if mode != MODE_PLAIN else np.ascontiguousarray(asr[:, :, :V])
        check_decode(f"B={B} mode={mode}", lm, o, a, mode, 0.5, starts, dev)
        case(f"decode launch B={B} mode={mode} ragged")
        gl, gs, _, _ = gpu_decode_launch(lm, a, mode, 0.5, starts, dev, lengths=lengths)
        ol, os_ = o.decode(a, mode, 0.5, starts, nthreads=NTHREADS, lengths=lengths)
        assert np.array_equal(gl, ol) and np.array_equal(gs, os_)


@pytest.mark.parametrize("V,B", [(40, 10000), (1000, 2400), (1024, 2400), (1025, 600), (1025, 2000), (2048, 1000),
                                 (2048, 1500)])
def test_decode_launch_row_placements(dev, V, B):
    """The whole decode with one wavefront per utterance keeps the ASR rows in
    registers up to V = 1024 when the model has 4-byte dense rows (these
    models do; with and without a last register chunk cut short by V, or with
    most chunks past V); above V = 1024 in two LDS buffers while every
    utterance is resident at once with them (on 256 CUs with 160 KiB of LDS
    each: 1792 at V = 1025, 1024 at V = 2048), else in one LDS buffer.  The
    cases cover each placement, and the four fusion modes on the register
    paths."""
    m, lm, o = pair(f"V{V}", lambda: generate_model(V, [V, 20000, 15000], 1.0, seed=V, bos_eos=True))
    T = 10
    starts = uniform_states(m, B, seed=B + 3)
    asr = asr_logprobs((B, T, V + 1), seed=B + 4, blank_boost=1.0)
    lengths = np.random.default_rng(B + 5).integers(0, T + 1, B).astype(np.int32)
    modes = (MODE_PLAIN, MODE_CTC, MODE_TRANSDUCER, MODE_AED) if V <= 1024 else (MODE_PLAIN, MODE_CTC)
    for mode in modes:
        a = asr if mode != MODE_PLAIN else np.ascontiguousarray(asr[:, :, :V])
        case(f"decode launch V={V} B={B} mode={mode} ragged")
        gl, gs, fin, _ = gpu_decode_launch(lm, a, mode, 0.5, starts, dev, lengths=lengths)
        assert lm.check_states() == 0
        ol, os_ = o.decode(a, mode, 0.5, starts, nthreads=NTHREADS, lengths=lengths)
        bad = np.argwhere(gl != ol)
        assert len(bad) == 0, f"labels differ first at {bad[0]}"
        assert np.array_equal(gs, os_)


@pytest.mark.parametrize("which", ["bigram", "zero_weight", "trigram"])
def test_decode_register_rows_dense_forms(dev, which):
    """Register-row decodes (2400 utterances at V = 1000) through both dense-row
    forms: a trigram model, whose 4-byte dense rows lead own bigrams to the
    row's base plus their rank; a bigram model, whose own entries lead to
    unigram states; and a trigram model with one bigram weight at +0.0 (sign
    bit clear), which gets no 4-byte rows, so the 8-byte rows serve it."""
    import struct
    V, B, T = 1000, 2400, 10
    if which == "bigram":
        m = generate_model(V, [V, 30000], 1.0, seed=11)
    else:
        m = generate_model(V, [V, 20000, 15000], 1.0, seed=12)
    order, tokens, W, Bo = m.to_list()
    if which == "zero_weight":
        W = W.copy()
        W[np.nonzero(order == 2)[0][5]] = 0.0
    lm = ng.NgpuLM(V, m.max_order, order, tokens, W, Bo, m.unk_logprob).upload(dev)
    o = Oracle(V, m.max_order, order, tokens, W, Bo, m.unk_logprob)
    hdr = struct.unpack_from("<IiiiqqQQQQQQ11i4x10QQiiQqiiQQ", lm.host_image()[:264].tobytes())
    assert (hdr[40] != 0) == (which != "zero_weight")
    starts = uniform_states(m, B, seed=13)
    asr = asr_logprobs((B, T, V + 1), seed=14, blank_boost=0.5)
    for mode in (MODE_PLAIN, MODE_CTC, MODE_TRANSDUCER):
        a = asr if mode != MODE_PLAIN else np.ascontiguousarray(asr[:, :, :V])
        case(f"decode launch register rows {which} mode={mode}")
        gl, gs, _, _ = gpu_decode_launch(lm, a, mode, 0.5, starts, dev)
        assert lm.check_states() == 0
        ol, os_ = o.decode(a, mode, 0.5, starts, nthreads=NTHREADS)
        bad = np.argwhere(gl != ol)
        assert len(bad) == 0, f"labels differ first at {bad[0]}"
        assert np.array_equal(gs, os_)


@pytest.mark.parametrize("V,B", [(1024, 32), (1024, 600), (1024, 2400), (1000, 2400)])
def test_decode_launch_time_major_view(dev, V, B):
    """The whole decode reads a time-major [T, B, C] buffer through a permuted
    [B, T, C] view (utterance stride C, frame stride B * C) whose rows carry
    padding past the classes: four wavefronts with LDS rows, and registers
    with and without a short last chunk, must read only the V (+ 1) classes
    of its own row."""
    if V == 1024:
        m, lm, o = model_pair("fourgram_200k")
    else:
        m, lm, o = pair(f"V{V}", lambda: generate_model(V, [V, 20000, 15000], 1.0, seed=V, bos_eos=True))
    T, pad = 9, 7
    starts = uniform_states(m, B, seed=B + 6)
    asr = asr_logprobs((B, T, V + 1), seed=B + 7, blank_boost=1.0)
    for mode in (MODE_PLAIN, MODE_CTC):
        C = V if mode == MODE_PLAIN else V + 1
        a = np.ascontiguousarray(asr[:, :, :C])
        tm = np.full((T, B, C + pad), 7.0, np.float32)     # padding above every log-probability
        tm[:, :, :C] = a.transpose(1, 0, 2)
        view = torch.from_numpy(tm).to(dev).permute(1, 0, 2)[:, :, :C]
        assert view.stride() == (C + pad, B * (C + pad), 1)
        st = torch.from_numpy(starts.copy()).to(dev)
        prev = torch.full((B,), V, dtype=torch.int32, device=dev) if mode == MODE_CTC else None
        case(f"decode launch time-major view V={V} B={B} mode={mode}")
        lab = lm.fused_greedy_decode(view, 0.5, st, prev, mode=mode)
        torch.cuda.synchronize()
        assert lm.check_states() == 0
        ol, os_ = o.decode(a, mode, 0.5, starts, nthreads=NTHREADS)
        assert np.array_equal(lab.cpu().numpy(), ol)
        assert np.array_equal(st.cpu().numpy(), os_[:, -1])


@pytest.mark.parametrize("B", [200, 2400])
def test_decode_launch_lambda_signs(dev, B):
    """Negative, zero and large lambda on the four-wavefront LDS path (200
    utterances) and the one-wavefront register path (2400): the CTC exclusion
    of the previous label must hold whatever sign the LM term takes."""
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    T = 12
    starts = uniform_states(m, B, seed=B + 8)
    asr = asr_logprobs((B, T, V + 1), seed=B + 9, blank_boost=0.5)
    for lam in (-0.7, 0.0, 3.0):
        for mode in (MODE_PLAIN, MODE_CTC):
            a = asr if mode != MODE_PLAIN else np.ascontiguousarray(asr[:, :, :V])
            case(f"decode launch B={B} lambda={lam} mode={mode}")
            gl, gs, _, _ = gpu_decode_launch(lm, a, mode, lam, starts, dev)
            assert lm.check_states() == 0
            ol, os_ = o.decode(a, mode, lam, starts, nthreads=NTHREADS)
            bad = np.argwhere(gl != ol)
            assert len(bad) == 0, f"labels differ first at {bad[0]}"
            assert np.array_equal(gs, os_)
            if B < 512:   # the per-frame step kernel too
                check_decode(f"lambda={lam} mode={mode}", lm, o, a, mode, lam, starts, dev)


def test_decode_launch_resumes_exactly(dev):
    """Two launches over frames [0, 40) and [40, 90), passing states and labels
    back, equal one decode over all 90 frames."""
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    B, T, cut = 24, 90, 40
    starts = uniform_states(m, B, seed=41)
    asr = asr_logprobs((B, T, V + 1), seed=42, blank_boost=2.0)
    case("decode launch resume")
    gl, gs, fin, fprev = gpu_decode_launch(lm, asr, MODE_CTC, 0.5, starts, dev)
    a1, s1, f1, p1 = gpu_decode_launch(lm, np.ascontiguousarray(asr[:, :cut]), MODE_CTC, 0.5, starts, dev)
    a2, s2, f2, p2 = gpu_decode_launch(lm, np.ascontiguousarray(asr[:, cut:]), MODE_CTC, 0.5, f1, dev, prev0=p1)
    assert np.array_equal(np.concatenate([a1, a2], 1), gl)
    assert np.array_equal(np.concatenate([s1, s2], 1), gs)
    assert np.array_equal(f2, fin) and np.array_equal(p2, fprev)


def test_decode_launch_bad_start_state(dev):
    m, lm, o = model_pair("trigram_v128")
    V = m.vocab_size
    asr = asr_logprobs((3, 7, V), seed=43)
    starts = np.array([2, m.num_states, 5], np.int32)
    case("decode launch with an out-of-range start state")
    gl, gs, fin, _ = gpu_decode_launch(lm, asr, MODE_PLAIN, 0.5, starts, dev)
    assert lm.check_states() == 1
    assert (gl[1] == -1).all() and (gs[1] == -1).all()
    ol, os_ = o.decode(asr[[0, 2]], MODE_PLAIN, 0.5, starts[[0, 2]])
    assert np.array_equal(gl[[0, 2]], ol) and np.array_equal(gs[[0, 2]], os_)


def test_fused_transducer_and_ctc_small(dev):
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    starts = uniform_states(m, 64, seed=5)
    asr = asr_logprobs((64, 40, V + 1), seed=6, blank_boost=3.0)
    check_decode("transducer 4-gram 200k", lm, o, asr, MODE_TRANSDUCER, 0.7, starts, dev)
    check_decode("ctc 4-gram 200k", lm, o, asr, MODE_CTC, 0.7, starts, dev)


def test_fused_ties_lambda_zero_and_all_blank(dev):
    m, lm, o = model_pair("trigram_v128")
    V = m.vocab_size
    B = 65
    starts = uniform_states(m, B, seed=8)
    asr = asr_logprobs((B, 6, V + 1), seed=9)
    asr[:, 0, :] = -3.0                       # full ties in frame 0
    asr[:5, 1, :] = -5.0
    asr[:5, 1, V] = -0.01                     # blank wins frame 1 for five rows
    asr[:, 2, 7] = asr[:, 2, 100] = 2.0       # two-way ties
    for mode in (MODE_PLAIN, MODE_CTC, MODE_TRANSDUCER):
        a = asr if mode != MODE_PLAIN else np.ascontiguousarray(asr[:, :, :V])
        for lam in (0.0, 0.5, -1.0, 4.0):
            check_decode(f"ties mode={mode} lambda={lam}", lm, o, a, mode, lam, starts, dev)
    # an all-blank utterance never moves its state
    allb = np.full((3, 10, V + 1), -9.0, np.float32)
    allb[:, :, V] = -0.001
    gl, gs = check_decode("all blank", lm, o, allb, MODE_CTC, 0.5, starts[:3], dev)
    assert (gl == V).all() and (gs == starts[:3, None]).all()


def _edge_frames(V, B):
    """Frames whose argmax hinges on -inf and on ties across lanes and stripes
    (tokens go four to a lane in stripes of 256)."""
    ninf = -np.inf
    asr = asr_logprobs((B, 8, V + 1), seed=13, blank_boost=0.5)
    asr[:, 0, :] = ninf                                    # every class at -inf
    asr[:, 1, :V] = ninf                                   # tokens at -inf, blank finite
    asr[:, 1, V] = -1.0
    for t, (i, j) in zip((2, 3, 4), ((252, 256), (5, 261), (767, 1023))):
        asr[:, t, :] = -9.0                                # two-way ties at the top:
        asr[:, t, i] = asr[:, t, j] = 5.0                  # lane 63 vs lane 0, same lane, same lane
    asr[:, 5, :] = ninf                                    # one finite token, blank -inf in half the rows
    asr[:, 5, 600] = -1.0
    asr[B // 2:, 5, V] = -2.0
    asr[:, 6, :] = -4.0                                    # -0 and +0 tie at the top
    asr[:, 6, 10] = -0.0
    asr[:, 6, 3] = 0.0
    return asr


@pytest.mark.parametrize("mode", [MODE_PLAIN, MODE_CTC, MODE_TRANSDUCER])
def test_fused_minus_inf_and_lane_ties(dev, mode):
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    B = 40
    asr = _edge_frames(V, B)
    if mode == MODE_PLAIN:
        asr = np.ascontiguousarray(asr[:, :, :V])
    starts = uniform_states(m, B, seed=14)
    for lam in (0.0, 0.5, -1.0):
        check_decode(f"edge frames mode={mode} lambda={lam}", lm, o, asr, mode, lam, starts, dev)
        case(f"edge frames decode launch mode={mode} lambda={lam}")
        gl, gs, _, _ = gpu_decode_launch(lm, asr, mode, lam, starts, dev)
        ol, os_ = o.decode(asr, mode, lam, starts, nthreads=NTHREADS)
        assert np.array_equal(gl, ol) and np.array_equal(gs, os_)
    if mode == MODE_PLAIN:
        assert (gl[:, 0] == 0).all()                       # all -inf: the first token
    else:
        assert (gl[:, 0] == 0).all() and (gl[:, 1] == V).all()


def test_aed_minus_inf_frames(dev):
    m, lm, o = aed_pair()
    V = m.vocab_size
    B = 24
    asr = _edge_frames(V, B)
    starts = uniform_states(m, B, seed=15)
    for lam in (0.0, 0.7):
        check_decode(f"aed edge frames lambda={lam}", lm, o, asr, MODE_AED, lam, starts, dev)
        gl, gs, _, _ = gpu_decode_launch(lm, asr, MODE_AED, lam, starts, dev)
        ol, os_ = o.decode(asr, MODE_AED, lam, starts, nthreads=NTHREADS)
        assert np.array_equal(gl, ol) and np.array_equal(gs, os_)
        assert (gl[:, 0] == 0).all() and (gl[:, 1] == V).all()


def test_max_vocabulary(dev):
    """V = 8192, the largest vocabulary the library takes: the LDS rows of
    every kernel at their largest."""
    m, lm, o = pair("V8192", lambda: generate_model(8192, [8192, 40000, 30000], 1.0, seed=8192))
    V = m.vocab_size
    assert V == 8192
    states = uniform_states(m, 700, seed=16)
    check_advance("V=8192", m, lm, o, states, dev)
    B, T = 20, 12
    asr = asr_logprobs((B, T, V + 1), seed=17, blank_boost=1.0)
    starts = states[:B]
    for mode in (MODE_PLAIN, MODE_CTC):
        a = asr if mode != MODE_PLAIN else np.ascontiguousarray(asr[:, :, :V])
        check_decode(f"V=8192 mode={mode}", lm, o, a, mode, 0.5, starts, dev)
        case(f"V=8192 decode launch mode={mode}")
        gl, gs, _, _ = gpu_decode_launch(lm, a, mode, 0.5, starts, dev)
        ol, os_ = o.decode(a, mode, 0.5, starts, nthreads=NTHREADS)
        assert np.array_equal(gl, ol) and np.array_equal(gs, os_)
    # above 512 utterances: one wavefront each, one LDS row buffer (98 KiB of LDS per workgroup)
    B2, T2 = 600, 6
    starts2 = uniform_states(m, B2, seed=18)
    asr2 = asr_logprobs((B2, T2, V + 1), seed=19, blank_boost=1.0)
    case(f"V=8192 decode launch B={B2}")
    gl, gs, _, _ = gpu_decode_launch(lm, asr2, MODE_CTC, 0.5, starts2, dev)
    ol, os_ = o.decode(asr2, MODE_CTC, 0.5, starts2, nthreads=NTHREADS)
    assert np.array_equal(gl, ol) and np.array_equal(gs, os_)
    case("V=8192 top-k k=20")
    a0 = np.ascontiguousarray(asr[:, 0, :V])
    tok, sc, nx = lm.fused_topk(torch.from_numpy(a0).to(dev), 0.5, 20, torch.from_numpy(starts).to(dev))
    torch.cuda.synchronize()
    assert lm.check_states() == 0
    ot, osc, onx = o.fused_topk(a0, 0.5, 20, starts)
    assert np.array_equal(tok.cpu().numpy(), ot) and np.array_equal(nx.cpu().numpy(), onx)
    assert np.abs(sc.cpu().numpy() - osc).max() <= TOL


def test_fused_strided_asr_rows(dev):
    """asr rows with a leading dimension larger than V + 1."""
    m, lm, o = model_pair("trigram_v128")
    V = m.vocab_size
    base = asr_logprobs((16, V + 1), seed=10, blank_boost=1.0)
    padded = np.full((16, V + 40), 7.0, np.float32)   # padding must never be read
    padded[:, :V + 1] = base
    case("fused with asr_ld = V + 40")
    st = torch.from_numpy(uniform_states(m, 16, seed=11)).to(dev)
    st0 = st.cpu().numpy().copy()
    prev = torch.full((16,), V, dtype=torch.int32, device=dev)
    tok = lm.fused_greedy_step(torch.from_numpy(padded).to(dev), 0.5, st, prev, mode=ng.NGPU_FUSION_CTC)
    torch.cuda.synchronize()
    o_st = st0.copy()
    o_prev = np.full(16, V, np.int32)
    o_tok = o.greedy_step(base, MODE_CTC, 0.5, o_st, o_prev)
    assert np.array_equal(tok.cpu().numpy(), o_tok)
    assert np.array_equal(st.cpu().numpy(), o_st)
    assert np.array_equal(prev.cpu().numpy(), o_prev)


@pytest.mark.parametrize("k", [1, 5, 32])
def test_fused_topk_4gram_200k(dev, k):
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    B = 50
    states = uniform_states(m, B, seed=51 + k)
    asr = asr_logprobs((B, V), seed=52 + k)
    asr[:3] = -7.0                            # full ties: lower index first
    case(f"fused top-k 4-gram 200k B={B} k={k}")
    tok, sc, nx = lm.fused_topk(torch.from_numpy(asr).to(dev), 0.6, k, torch.from_numpy(states).to(dev))
    torch.cuda.synchronize()
    assert lm.check_states() == 0
    ot, osc, onx = o.fused_topk(asr, 0.6, k, states)
    assert np.array_equal(tok.cpu().numpy(), ot)
    assert np.array_equal(nx.cpu().numpy(), onx)
    assert np.abs(sc.cpu().numpy() - osc).max() <= TOL


@pytest.mark.parametrize("lam", [0.0, 0.6])
def test_fused_topk_minus_inf_and_ties(dev, lam):
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    B, k = 8, 12
    states = uniform_states(m, B, seed=61)
    asr = asr_logprobs((B, V), seed=62)
    asr[0] = -np.inf                                   # nothing finite: lowest indices in order
    asr[1] = -np.inf                                   # three finite tokens, then the lowest untaken
    asr[1, [900, 5, 300]] = [-1.0, -2.0, -3.0]
    asr[2] = -7.0                                      # full ties
    asr[3] = -9.0                                      # ties across lanes and stripes
    asr[3, [260, 4, 256, 252, 1023, 767]] = 5.0
    asr[4, :] = -np.inf                                # finite tokens fewer than k, spread over lanes
    asr[4, ::97] = -0.5
    case(f"fused top-k -inf rows and ties lambda={lam}")
    tok, sc, nx = lm.fused_topk(torch.from_numpy(asr).to(dev), lam, k, torch.from_numpy(states).to(dev))
    torch.cuda.synchronize()
    assert lm.check_states() == 0
    ot, osc, onx = o.fused_topk(asr, lam, k, states)
    assert np.array_equal(tok.cpu().numpy(), ot)
    assert np.array_equal(nx.cpu().numpy(), onx)
    g = sc.cpu().numpy()
    assert np.array_equal(np.isinf(g), np.isinf(osc))
    fin = np.isfinite(osc)
    assert np.abs(g[fin] - osc[fin]).max() <= TOL
    assert ot[0].tolist() == list(range(k))
    if lam == 0.0:
        assert ot[3, :6].tolist() == [4, 252, 256, 260, 767, 1023]


@pytest.mark.parametrize("V", [128, 500, 700])
def test_fused_topk_vocab_sizes(dev, V):
    """Vocabularies of one, two and three 256-token stripes per lane (the
    register top-k), with -inf rows and ties."""
    m, lm, o = pair(f"topk V{V}", lambda: generate_model(V, [V, 6 * V, 6 * V], 1.0, seed=V + 7))
    B, k = 40, 12
    states = uniform_states(m, B, seed=V + 8)
    asr = asr_logprobs((B, V), seed=V + 9)
    asr[0] = -np.inf
    asr[1] = -4.0
    asr[2, :] = -np.inf
    asr[2, ::37] = -1.0
    for lam in (0.0, 0.6):
        case(f"fused top-k V={V} k={k} lambda={lam}")
        tok, sc, nx = lm.fused_topk(torch.from_numpy(asr).to(dev), lam, k, torch.from_numpy(states).to(dev))
        torch.cuda.synchronize()
        assert lm.check_states() == 0
        ot, osc, onx = o.fused_topk(asr, lam, k, states)
        assert np.array_equal(tok.cpu().numpy(), ot)
        assert np.array_equal(nx.cpu().numpy(), onx)
        g = sc.cpu().numpy()
        fin = np.isfinite(osc)
        assert np.array_equal(np.isfinite(g), fin) and np.abs(g[fin] - osc[fin]).max() <= TOL


def test_sync_check(dev):
    """ngpu_lm_sync_check: NGPU_E_BAD_STATE after queries that met out-of-range
    states (the count clears), NGPU_OK after clean ones."""
    m, lm, o = model_pair("trigram_v128")
    states = uniform_states(m, 12, seed=90)
    states[[2, 7]] = [-1, m.num_states]
    case("sync check")
    run_advance(lm, states, dev)
    with pytest.raises(ng.NgpuError) as e:
        lm.sync_check()
    assert e.value.code == -12
    lm.sync_check()                      # cleared
    run_advance(lm, uniform_states(m, 12, seed=91), dev)
    lm.sync_check()


@pytest.mark.parametrize("k", [6, 8, 64, 100, 128, 256])
def test_fused_topk_large_k(dev, k):
    """The threshold selection (every k at V <= 1024) at larger k: rows of full
    ties, -inf rows, rows with fewer finite tokens than k, rows whose fused
    values are coarsely quantised so that many tokens tie across lanes and
    stripes, and ordinary rows.  k = 64 and 128 are the largest k whose search
    starts from the smallest lane maximum and lane second-maximum; above 128 it
    starts from no lower bound."""
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    B = 24
    states = uniform_states(m, B, seed=70 + k)
    asr = asr_logprobs((B, V), seed=71 + k)
    asr[0] = -3.0
    asr[1] = -np.inf
    asr[2] = -np.inf
    asr[2, ::11] = -1.0                       # 94 finite tokens
    asr[3:8] = np.round(asr[3:8] * 2) / 2     # many exact ties at lambda = 0
    for lam in (0.0, 0.6):
        case(f"fused top-k large k={k} lambda={lam}")
        tok, sc, nx = lm.fused_topk(torch.from_numpy(asr).to(dev), lam, k, torch.from_numpy(states).to(dev))
        torch.cuda.synchronize()
        assert lm.check_states() == 0
        ot, osc, onx = o.fused_topk(asr, lam, k, states)
        assert np.array_equal(tok.cpu().numpy(), ot)
        assert np.array_equal(nx.cpu().numpy(), onx)
        g = sc.cpu().numpy()
        fin = np.isfinite(osc)
        assert np.array_equal(np.isfinite(g), fin) and np.abs(g[fin] - osc[fin]).max() <= TOL
        assert ot[0].tolist() == list(range(k)) or lam != 0.0


def test_fused_topk_k_equals_vocab(dev):
    """k = V on a V = 128 model: every token once, in the definition's order."""
    m, lm, o = model_pair("trigram_v128")
    V = m.vocab_size
    B = 16
    states = uniform_states(m, B, seed=81)
    asr = asr_logprobs((B, V), seed=82)
    asr[0] = -2.0
    asr[1, :] = -np.inf
    asr[1, 5::9] = 0.0
    case(f"fused top-k k=V={V}")
    tok, sc, nx = lm.fused_topk(torch.from_numpy(asr).to(dev), 0.4, V, torch.from_numpy(states).to(dev))
    torch.cuda.synchronize()
    ot, osc, onx = o.fused_topk(asr, 0.4, V, states)
    assert np.array_equal(tok.cpu().numpy(), ot) and np.array_equal(nx.cpu().numpy(), onx)
    assert (np.sort(tok.cpu().numpy(), axis=1) == np.arange(V)).all()
    g = sc.cpu().numpy()
    fin = np.isfinite(osc)
    assert np.array_equal(np.isfinite(g), fin) and np.abs(g[fin] - osc[fin]).max() <= TOL


def test_fused_topk_odd_vocab_and_bad_state(dev):
    m, lm, o = pair("V1025N4", lambda: generate_model(1025, [1025, 6150, 6150, 6150], 1.0, seed=1029))
    V = m.vocab_size
    states = uniform_states(m, 9, seed=53)
    states[4] = -3
    asr = asr_logprobs((9, V), seed=54)
    case("fused top-k V=1025 k=7 with a bad state")
    tok, sc, nx = lm.fused_topk(torch.from_numpy(asr).to(dev), 1.1, 7, torch.from_numpy(states).to(dev))
    torch.cuda.synchronize()
    assert lm.check_states() == 1
    t, s_, n = tok.cpu().numpy(), sc.cpu().numpy(), nx.cpu().numpy()
    assert (t[4] == -1).all() and np.isnan(s_[4]).all() and (n[4] == -1).all()
    good = [0, 1, 2, 3, 5, 6, 7, 8]
    ot, osc, onx = o.fused_topk(asr[good], 1.1, 7, states[good])
    assert np.array_equal(t[good], ot) and np.array_equal(n[good], onx)
    assert np.abs(s_[good] - osc).max() <= TOL


def aed_pair():
    return pair("aed", lambda: generate_model(1024, [1024, 20000, 30000, 20000], 1.05, seed=77, bos_eos=True))


def test_aed_advance_and_final_weights(dev):
    m, lm, o = aed_pair()
    assert lm.start_state == o.start_state
    states = np.concatenate([[lm.start_state, 0], uniform_states(m, 3000, seed=78)]).astype(np.int32)
    check_advance("aed model", m, lm, o, states, dev)
    case("final weights")
    fin = lm.final_weights(torch.from_numpy(states).to(dev))
    torch.cuda.synchronize()
    assert lm.check_states() == 0
    assert np.array_equal(fin.cpu().numpy(), o.final(states))


def test_aed_greedy_step_and_decode(dev):
    m, lm, o = aed_pair()
    V = m.vocab_size
    B, T = 48, 60
    asr = asr_logprobs((B, T, V + 1), seed=79, blank_boost=1.5)     # class V is <eos>
    starts = np.full(B, lm.start_state, np.int32)
    starts[B // 2:] = uniform_states(m, B - B // 2, seed=80)
    for lam in (0.0, 0.6, 2.0):
        check_decode(f"aed per-frame lambda={lam}", lm, o, asr, MODE_AED, lam, starts, dev)
        case(f"aed decode launch lambda={lam}")
        gl, gs, fin, _ = gpu_decode_launch(lm, asr, MODE_AED, lam, starts, dev)
        ol, os_ = o.decode(asr, MODE_AED, lam, starts, nthreads=NTHREADS)
        assert np.array_equal(gl, ol) and np.array_equal(gs, os_)
        print(f"  aed lambda={lam}: <eos> labels {(gl == V).mean():.3f}", flush=True)


def test_aed_mode_needs_final_weights(dev):
    m, lm, o = model_pair("trigram_v128")
    asr = torch.zeros((2, m.vocab_size + 1), device=dev)
    st = torch.zeros(2, dtype=torch.int32, device=dev)
    with pytest.raises(ng.NgpuError):
        lm.fused_greedy_step(asr, 0.5, st, mode=ng.NGPU_FUSION_AED)
    with pytest.raises(ng.NgpuError):
        lm.final_weights(st)


def test_graph_capture_replays_match_eager(dev):
    """The per-frame steps and an advance captured in one HIP graph (the paper
    runs its decoding steps in CUDA graphs) give the eager results on every
    replay, with eager work in between."""
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    B, T = 32, 12
    asr_np = asr_logprobs((T, B, V + 1), seed=91, blank_boost=2.0)
    starts = uniform_states(m, B, seed=92)
    asr = torch.from_numpy(asr_np).to(dev)
    st = torch.from_numpy(starts).to(dev)
    prev = torch.full((B,), V, dtype=torch.int32, device=dev)
    toks = torch.empty((T, B), dtype=torch.int32, device=dev)
    sc = torch.empty((B, V), dtype=torch.float32, device=dev)
    nx = torch.empty((B, V), dtype=torch.int32, device=dev)
    st0 = st.clone()
    # a whole-decode launch and a top-k on their own buffers
    dasr = torch.from_numpy(np.ascontiguousarray(asr_np.transpose(1, 0, 2))).to(dev)
    dst = torch.empty(B, dtype=torch.int32, device=dev)
    dprev = torch.empty(B, dtype=torch.int32, device=dev)
    dlab = torch.empty((B, T), dtype=torch.int32, device=dev)
    ktok = torch.empty((B, 6), dtype=torch.int32, device=dev)
    ksc = torch.empty((B, 6), dtype=torch.float32, device=dev)
    knx = torch.empty((B, 6), dtype=torch.int32, device=dev)

    def body():
        for t in range(T):
            lm.fused_greedy_step(asr[t], 0.5, st, prev, mode=ng.NGPU_FUSION_CTC, tokens=toks[t])
        lm.advance(st, sc, nx)
        dst.copy_(st0)
        dprev.fill_(V)
        lm.fused_greedy_decode(dasr, 0.5, dst, dprev, mode=ng.NGPU_FUSION_CTC, labels=dlab)
        lm.fused_topk(asr[0, :, :V], 0.7, 6, st, tokens=ktok, scores=ksc, next_states=knx)

    # eager reference
    body()
    torch.cuda.synchronize()
    ref = [x.clone() for x in (toks, st, prev, sc, nx, dst, dprev, dlab, ktok, ksc, knx)]
    case("graph capture of 12 fused steps and one advance")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                 # warm the libraries on the capture stream
        st.copy_(st0)
        prev.fill_(V)
        body()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    st.copy_(st0)
    prev.fill_(V)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        body()
    for r in range(4):
        st.copy_(st0)
        prev.fill_(V)
        toks.fill_(-9)
        sc.fill_(float("nan"))
        dlab.fill_(-9)
        ktok.fill_(-9)
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip((toks, st, prev, sc, nx, dst, dprev, dlab, ktok, ksc, knx), ref):
            assert torch.equal(a, b), f"replay {r} differs"
        _ = lm.advance(st)                        # eager work between replays
        torch.cuda.synchronize()
    assert lm.check_states() == 0
    ol, os_ = o.decode(np.ascontiguousarray(asr_np.transpose(1, 0, 2)), MODE_CTC, 0.5, starts)
    assert np.array_equal(ref[0].cpu().numpy().T, ol)
    assert np.array_equal(ref[7].cpu().numpy(), ol)           # the whole-decode launch
    ot, _, onx = o.fused_topk(np.ascontiguousarray(asr_np[0, :, :V]), 0.7, 6, ref[1].cpu().numpy())
    assert np.array_equal(ref[8].cpu().numpy(), ot) and np.array_equal(ref[10].cpu().numpy(), onx)


def test_concurrent_streams_match_sequential(dev):
    """Queries on one uploaded model from four streams at once (advance, a
    whole decode, per-frame steps and top-k, each on its own buffers) give
    what they give one after another: the library keeps no per-call state
    besides the status count."""
    m, lm, o = model_pair("fourgram_200k")
    V = m.vocab_size
    B, T = 96, 20
    st_adv = torch.from_numpy(uniform_states(m, 700, seed=61)).to(dev)
    starts = uniform_states(m, B, seed=62)
    asr = torch.from_numpy(asr_logprobs((B, T, V + 1), seed=63, blank_boost=1.0)).to(dev)
    rows = [asr[:, t, :].contiguous() for t in range(T)]

    def run(streams):
        out = {}
        with torch.cuda.stream(streams[0]):
            out["adv"] = lm.advance(st_adv, stream=streams[0])
        with torch.cuda.stream(streams[1]):
            st = torch.from_numpy(starts).to(dev)
            prev = torch.full((B,), V, dtype=torch.int32, device=dev)
            out["dec"] = (lm.fused_greedy_decode(asr, 0.5, st, prev, mode=ng.NGPU_FUSION_CTC, stream=streams[1]), st)
        with torch.cuda.stream(streams[2]):
            st2 = torch.from_numpy(starts).to(dev)
            prev2 = torch.full((B,), V, dtype=torch.int32, device=dev)
            toks = [lm.fused_greedy_step(r, 0.5, st2, prev2, mode=ng.NGPU_FUSION_CTC, stream=streams[2]).clone()
                    for r in rows]
            out["step"] = (torch.stack(toks, 1), st2)
        with torch.cuda.stream(streams[3]):
            out["topk"] = lm.fused_topk(rows[0][:, :V].contiguous(), 0.5, 8, torch.from_numpy(starts).to(dev),
                                        stream=streams[3])
        torch.cuda.synchronize()
        return out

    case("four streams at once against one stream")
    main = torch.cuda.current_stream()
    seq = run([main] * 4)
    par = run([torch.cuda.Stream() for _ in range(4)])
    assert lm.check_states() == 0
    assert torch.equal(seq["adv"][0], par["adv"][0]) and torch.equal(seq["adv"][1], par["adv"][1])
    assert torch.equal(seq["dec"][0], par["dec"][0]) and torch.equal(seq["dec"][1], par["dec"][1])
    assert torch.equal(seq["step"][0], par["step"][0]) and torch.equal(seq["step"][1], par["step"][1])
    assert all(torch.equal(a, b) for a, b in zip(seq["topk"], par["topk"]))
    # and the decode and the per-frame steps agree with each other and the oracle
    assert torch.equal(par["dec"][0], par["step"][0])
    ol, _ = o.decode(asr.cpu().numpy(), MODE_CTC, 0.5, starts, nthreads=NTHREADS)
    assert np.array_equal(par["dec"][0].cpu().numpy(), ol)


def test_fused_zero_sizes(dev):
    """B = 0 (and T = 0 for the decode) launch nothing and change nothing."""
    m, lm, o = model_pair("trigram_v128")
    V = m.vocab_size
    case("fused entry points with B = 0 / T = 0")
    empty_asr = torch.empty((0, V + 1), device=dev)
    st0 = torch.empty(0, dtype=torch.int32, device=dev)
    assert lm.fused_greedy_step(empty_asr, 0.5, st0, mode=ng.NGPU_FUSION_CTC,
                                prev=torch.empty(0, dtype=torch.int32, device=dev)).numel() == 0
    tok, sc, nx = lm.fused_topk(torch.empty((0, V), device=dev), 0.5, 3, st0)
    assert tok.shape == (0, 3) and sc.shape == (0, 3) and nx.shape == (0, 3)
    st = torch.tensor([3, 5], dtype=torch.int32, device=dev)
    prev = torch.full((2,), V, dtype=torch.int32, device=dev)
    lab = lm.fused_greedy_decode(torch.empty((2, 0, V + 1), device=dev), 0.5, st, prev, mode=ng.NGPU_FUSION_CTC)
    torch.cuda.synchronize()
    assert lab.shape == (2, 0) and st.tolist() == [3, 5] and prev.tolist() == [V, V]
    assert lm.check_states() == 0


def test_batches_beyond_the_dispatch_limit_are_rejected(dev):
    """B above NGPU_LM_MAX_BATCH (2^26 - 256) is an error for every batched call,
    before any pointer is read."""
    import ctypes
    m, lm, o = model_pair("trigram_v128")
    big = (1 << 26) - 255
    buf = torch.zeros(1024, dtype=torch.int32, device=dev)
    p = ctypes.c_void_p(buf.data_ptr())
    L, h = lm._lib, lm._h
    case("batches beyond the dispatch limit")
    assert L.ngpu_lm_advance(h, p, big, p, p, None) == -1
    assert L.ngpu_lm_fused_greedy_step(h, p, big, m.vocab_size + 1, 1, ctypes.c_float(0.5), p, p, p, None) == -1
    assert L.ngpu_lm_fused_topk(h, p, big, m.vocab_size, ctypes.c_float(0.5), 3, p, p, p, p, None) == -1
    assert L.ngpu_lm_fused_greedy_decode(h, p, big, 1, m.vocab_size + 1, m.vocab_size + 1, None, 1,
                                         ctypes.c_float(0.5), p, p, p, None, None) == -1
    assert L.ngpu_lm_final_weights(h, p, big, p, None) in (-1,)   # no </s>: rejected either way


def test_binding_rejects_short_asr_rows(dev):
    """The binding checks the class width the C-ABI cannot see: V classes, plus
    blank (or <eos>) outside plain fusion."""
    m, lm, o = model_pair("trigram_v128")
    V = m.vocab_size
    st = torch.zeros(4, dtype=torch.int32, device=dev)
    prev = torch.full((4,), V, dtype=torch.int32, device=dev)
    case("binding: short asr rows")
    with pytest.raises(ValueError):
        lm.fused_greedy_step(torch.zeros((4, V), device=dev), 0.5, st, prev, mode=ng.NGPU_FUSION_CTC)
    with pytest.raises(ValueError):
        lm.fused_greedy_decode(torch.zeros((4, 3, V), device=dev), 0.5, st, prev, mode=ng.NGPU_FUSION_CTC)
    with pytest.raises(ValueError):
        lm.fused_greedy_decode(torch.zeros((4, 3, V + 1), device=dev)[:, :, :V - 1], 0.5, st)
    with pytest.raises(ValueError):
        lm.fused_topk(torch.zeros((4, V - 1), device=dev), 0.5, 2, st)
    # plain fusion takes V classes; wider rows are fine
    lm.fused_greedy_step(torch.zeros((4, V), device=dev), 0.5, st)
    lm.fused_greedy_decode(torch.zeros((4, 3, V + 9), device=dev), 0.5, st, prev, mode=ng.NGPU_FUSION_CTC)
    torch.cuda.synchronize()
    assert lm.check_states() == 0


def test_fused_out_of_range_state(dev):
    m, lm, o = model_pair("trigram_v128")
    V = m.vocab_size
    case("fused with an out-of-range state")
    st = torch.tensor([3, m.num_states + 5, 0], dtype=torch.int32, device=dev)
    asr = torch.from_numpy(asr_logprobs((3, V), seed=12)).to(dev)
    tok = lm.fused_greedy_step(asr, 0.5, st)
    torch.cuda.synchronize()
    assert lm.check_states() == 1
    t = tok.cpu().numpy()
    assert t[1] == -1 and int(st[1]) == m.num_states + 5
    o_st = np.array([3, 0], np.int32)
    o_tok = o.greedy_step(asr.cpu().numpy()[[0, 2]], MODE_PLAIN, 0.5, o_st)
    assert t[[0, 2]].tolist() == o_tok.tolist()
