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


def seed_for(index: int) -> int:
    return SEED_BASE + index


@dataclass(frozen=True)
class ConfigSpec:
    index: int
    name: str
    vocab_size: int
    counts: Tuple[int, ...]
    zipf_s: float
    batch: int
    steps: int = 0            # greedy steps (PLAIN) or frames (CTC)
    lam: float = 0.5
    mode: str = "advance"     # advance | plain | ctc
    n_phrases: int = 0
    blank_boost: float = 0.0
    model_of: Optional[int] = None   # reuse another config's model

    @property
    def max_order(self) -> int:
        return len(self.counts)


CONFIGS = {
    1: ConfigSpec(1, "tiny trigram V=128", 128, (128, 2000, 3000), 1.1,
                  batch=4, steps=50, mode="plain"),
    2: ConfigSpec(2, "4-gram V=1024 200k n-grams", 1024, (1024, 60000, 80000, 59000), 1.05,
                  batch=32, steps=200, mode="plain"),
    3: ConfigSpec(3, "6-gram context-biasing V=1024 2M n-grams", 1024,
                  (1024, 462000, 740000, 555000, 205000, 36976), 1.05,
                  batch=128, n_phrases=5000),
    4: ConfigSpec(4, "6-gram V=1024 20M n-grams", 1024,
                  (1024, 800000, 6500000, 7800000, 3900000, 998976), 1.0, batch=512),
    5: ConfigSpec(5, "fused greedy CTC on the 20M 6-gram", 1024,
                  (1024, 800000, 6500000, 7800000, 3900000, 998976), 1.0,
                  batch=256, steps=1000, mode="ctc", blank_boost=4.0, model_of=4),
}


def make_phrases(spec: ConfigSpec, rng: np.random.Generator):
    """Synthetic 3..8-token phrases of Zipf tokens (context-biasing word lists)."""
    V = spec.vocab_size
    perm = rng.permutation(V)
    z = 1.0 / np.arange(1, V + 1, dtype=np.float64) ** spec.zipf_s
    p = np.empty(V)
    p[perm] = z / z.sum()
    lens = rng.integers(3, 9, size=spec.n_phrases)
    return [rng.choice(V, size=int(L), p=p) for L in lens]


_MODEL_CACHE = {}


def make_config_model(index: int, cache: bool = True) -> NgramModel:
    """Model of config ``index`` (1..5); config 5 reuses config 4's model."""
    spec = CONFIGS[index]
    if spec.model_of is not None:
        return make_config_model(spec.model_of, cache)
    if cache and index in _MODEL_CACHE:
        return _MODEL_CACHE[index]
    phrases = None
    if spec.n_phrases:
        phrases = make_phrases(spec, np.random.default_rng(seed_for(index) + 7919))
    m = generate_model(spec.vocab_size, spec.counts, spec.zipf_s, seed_for(index), phrases)
    if cache:
        _MODEL_CACHE[index] = m
    return m
