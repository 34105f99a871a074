"""The five synthetic workloads, shaped like the paper's setting.

The paper's LMs are token-level KenLM models over a 1024-token BPE vocabulary,
up to order 10, from under 100 MB up to 1.5 GB on the GPU (Section 3.1).  Those
models and their text corpora are not available, so these seeded synthetic
models stand in for them with the same vocabulary, orders and size range.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np

from .ngram import NgramModel, generate_model

SEED_BASE = 20250522857


@dataclass(frozen=True)
class Workload:
    key: str
    name: str
    seed: int
    vocab_size: int
    counts: Tuple[int, ...]
    zipf_s: float
    batch: int
    steps: int = 0            # greedy steps (PLAIN) or frames (CTC)
    lam: float = 0.5
    mode: str = "advance"     # advance | plain | ctc
    n_phrases: int = 0
    blank_boost: float = 0.0
    model_of: Optional[str] = None   # reuse another workload's model

    @property
    def max_order(self) -> int:
        return len(self.counts)


_COUNTS_20M = (1024, 800000, 6500000, 7800000, 3900000, 998976)

WORKLOADS = {w.key: w for w in (
    Workload("trigram_v128", "trigram V=128, 5k n-grams, 4 hypotheses x 50 plain steps", SEED_BASE + 1, 128,
             (128, 2000, 3000), 1.1, batch=4, steps=50, mode="plain"),
    Workload("fourgram_200k", "4-gram V=1024, 200k n-grams, 32 hypotheses x 200 plain steps", SEED_BASE + 2,
             1024, (1024, 60000, 80000, 59000), 1.05, batch=32, steps=200, mode="plain"),
    Workload("sixgram_2m_phrases", "6-gram context-biasing V=1024, 2M n-grams with 5000 phrases, 128 states",
             SEED_BASE + 3, 1024, (1024, 462000, 740000, 555000, 205000, 36976), 1.05, batch=128, n_phrases=5000),
    Workload("sixgram_20m", "6-gram V=1024, 20M n-grams, 512 uniform states", SEED_BASE + 4, 1024, _COUNTS_20M,
             1.0, batch=512),
    Workload("ctc_b256_t1000", "greedy CTC fusion on the 20M 6-gram, 256 utterances x 1000 frames", SEED_BASE + 5,
             1024, _COUNTS_20M, 1.0, batch=256, steps=1000, mode="ctc", blank_boost=4.0, model_of="sixgram_20m"),
)}


def seed_for(key: str) -> int:
    """The seed of a workload's inputs."""
    return WORKLOADS[key].seed


def make_phrases(spec: Workload, rng: np.random.Generator):
    """Synthetic 3..8-token phrases of Zipf tokens (context-biasing word lists)."""
    V = spec.vocab_size
    perm = rng.permutation(V)
    z = 1.0 / np.arange(1, V + 1, dtype=np.float64) ** spec.zipf_s
    p = np.empty(V)
    p[perm] = z / z.sum()
    lens = rng.integers(3, 9, size=spec.n_phrases)
    return [rng.choice(V, size=int(L), p=p) for L in lens]


_MODEL_CACHE = {}


def make_model(key: str, cache: bool = True) -> NgramModel:
    """The model of workload ``key`` (the CTC workload reuses the 20M 6-gram's)."""
    spec = WORKLOADS[key]
    if spec.model_of is not None:
        return make_model(spec.model_of, cache)
    if cache and key in _MODEL_CACHE:
        return _MODEL_CACHE[key]
    phrases = None
    if spec.n_phrases:
        phrases = make_phrases(spec, np.random.default_rng(spec.seed + 7919))
    m = generate_model(spec.vocab_size, spec.counts, spec.zipf_s, spec.seed, phrases)
    if cache:
        _MODEL_CACHE[key] = m
    return m
