"""Seeded synthetic inputs shared by the tests, ``bench.py`` and the oracle checks.

This package builds random n-gram language models that are closed (every listed
n-gram's prefix and suffix are listed) and normalised by construction (every
context's conditional distribution sums to one once the backoff rule is
applied), plus query workloads: state batches and ASR log-probability tensors.

It holds model *construction* only: explicit log-probabilities and the backoff
weights that make each context normalised.  It never evaluates the backoff
query (no chain walk, no scoring of a context), so neither the GPU library nor
the oracle shares arithmetic with it.
"""

from .ngram import NgramModel, generate_model, lookup_ids, state_ids_of
from .configs import WORKLOADS, Workload, make_model, seed_for
from .workloads import (asr_logprobs, uniform_states, phrase_states,
                        tiny_model, pruned_list)
from .arpa import write_arpa, write_arpa_list, bpe_like_vocab

__all__ = [
    "NgramModel", "generate_model", "lookup_ids", "state_ids_of",
    "WORKLOADS", "Workload", "make_model", "seed_for",
    "asr_logprobs", "uniform_states", "phrase_states", "tiny_model",
    "write_arpa", "write_arpa_list", "bpe_like_vocab", "pruned_list",
]
