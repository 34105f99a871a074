"""Seeded query workloads: state batches and ASR log-probability tensors."""

from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from .ngram import NgramModel, generate_model, state_ids_of


def uniform_states(model: NgramModel, B: int, seed: int) -> np.ndarray:
    """``B`` canonical state ids drawn uniformly from ``[0, S)`` (every state is reachable)."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, model.num_states, size=B, dtype=np.int64).astype(np.int32)


def phrase_states(model: NgramModel, B: int, seed: int, depth: Optional[int] = None) -> np.ndarray:
    """States whose context is a length-``depth`` window of a phrase (deep backoff chains).

    Feeding ``noise token + phrase prefix`` (prefix length >= depth) from the
    start state ends in the state of the prefix's last ``depth`` tokens, because
    every phrase substring of length < N is listed; this returns those states.
    """
    if not model.phrases:
        raise ValueError("model has no phrases")
    depth = depth or (model.max_order - 1)
    rng = np.random.default_rng(seed)
    long = [p for p in model.phrases if len(p) >= depth]
    pick = rng.integers(0, len(long), size=B)
    ctx = []
    for i in pick:
        p = long[int(i)]
        end = int(rng.integers(depth, len(p) + 1))
        ctx.append(p[end - depth:end])
    ids = state_ids_of(model, np.stack(ctx))
    assert (ids >= 0).all()
    return ids


def asr_logprobs(shape: Sequence[int], seed: int, sigma: float = 3.0,
                 blank_boost: float = 0.0, chunk_rows: int = 65536) -> np.ndarray:
    """fp32 ``log_softmax`` over the last axis of ``N(0, sigma)`` logits.

    With ``blank_boost`` the last class (the CTC blank) gets ``+blank_boost``
    added to its logit before the softmax.  Computed in float64, stored fp32.
    """
    shape = tuple(int(s) for s in shape)
    C = shape[-1]
    rows = int(np.prod(shape[:-1]))
    rng = np.random.default_rng(seed)
    out = np.empty((rows, C), np.float32)
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        x = rng.standard_normal((r1 - r0, C), dtype=np.float32).astype(np.float64) * sigma
        if blank_boost:
            x[:, -1] += blank_boost
        mx = x.max(axis=1, keepdims=True)
        lse = mx + np.log(np.exp(x - mx).sum(axis=1, keepdims=True))
        out[r0:r1] = (x - lse).astype(np.float32)
    return out.reshape(shape)


def tiny_model(V: int, N: int, seed: int, fill: float = 0.5, n_unigrams: Optional[int] = None,
               zipf_s: float = 1.0) -> NgramModel:
    """A small random model for brute-force checks: ``fill`` of the candidates at each order."""
    counts = [n_unigrams if n_unigrams is not None else V]
    rng = np.random.default_rng(seed + 1)
    prev_count = counts[0]
    for k in range(2, N + 1):
        # an upper bound on candidates is prev_count * V; the sampler clamps to the real set
        c = max(1, int(fill * prev_count * min(V, counts[0]) * (0.6 if k > 2 else 1.0)))
        c = int(rng.integers(max(1, c // 2), c + 1))
        counts.append(c)
        prev_count = c
    return generate_model(V, counts, zipf_s, seed)


def pruned_list(model: NgramModel, drop: float, seed: int, drop_unigrams: int = 0):
    """The model's n-gram list with a random fraction `drop` of the n-grams of
    orders 2 .. N-1 removed (and `drop_unigrams` unigrams, for models with an
    <unk> weight): a list that is not closed, as a pruned ARPA model can be.
    Returns (order, tokens, logprob, backoff)."""
    o, t, W, B = model.to_list()
    rng = np.random.default_rng(seed)
    keep = np.ones(len(o), bool)
    mid = np.flatnonzero((o >= 2) & (o < model.max_order))
    keep[rng.choice(mid, int(drop * len(mid)), replace=False)] = False
    if drop_unigrams:
        uni = np.flatnonzero((o == 1) & (t[:, 0] < model.vocab_size))
        keep[rng.choice(uni, drop_unigrams, replace=False)] = False
    return o[keep], t[keep], W[keep], B[keep]
