"""Test infrastructure: the backoff rule stated on raw histories, for tiny models.

This is a second, independent statement of what a query computes, written
against token histories rather than states (Section 2.1): the score of token v
after history h is the recursion W(v | c) = B(c) + W(v | c[1:]) started from
the last N-1 tokens of h, with B(c) = 0 for an unlisted context and the <unk>
weight at the empty context; the state after h+(v) is the longest suffix of
h+(v), at most N-1 tokens long, that is a listed context.  It evaluates the
recursion right to left in Python floats (double), so it agrees with the
oracle's double result to rounding, not bit for bit.
"""

from __future__ import annotations

import math
from typing import Dict, Tuple


class BruteForce:
    def __init__(self, vocab_size, max_order, order, tokens, logprob, backoff,
                 unk_logprob=float("nan"), eos=None):
        self.V = int(vocab_size)
        self.N = int(max_order)
        self.unk = float(unk_logprob)
        self.eos = eos              # id of </s>: n-grams ending in it are no contexts
        self.W: Dict[Tuple[int, ...], float] = {}
        self.B: Dict[Tuple[int, ...], float] = {}
        for i in range(len(order)):
            g = tuple(int(t) for t in tokens[i][: int(order[i])])
            self.W[g] = float(logprob[i])
            self.B[g] = float(backoff[i])

    @classmethod
    def from_model(cls, model):
        eos = model.vocab_size + 1 if getattr(model, "bos_eos", False) else None
        return cls(model.vocab_size, model.max_order, *model.to_list(), model.unk_logprob, eos=eos)

    def _rec(self, ctx: Tuple[int, ...], v: int) -> float:
        if ctx + (v,) in self.W:
            return self.W[ctx + (v,)]
        if not ctx:
            if math.isnan(self.unk):
                raise KeyError("token without unigram and no <unk>")
            return self.unk
        return self.B.get(ctx, 0.0) + self._rec(ctx[1:], v)

    def score(self, history, v: int) -> float:
        h = tuple(int(t) for t in history)
        ctx = h[max(0, len(h) - (self.N - 1)):] if self.N > 1 else ()
        return self._rec(ctx, int(v))

    def is_context(self, c: Tuple[int, ...]) -> bool:
        if len(c) and self.eos is not None and c[-1] == self.eos:
            return False
        return len(c) == 0 or (len(c) < self.N and c in self.W)

    def state_context(self, history) -> Tuple[int, ...]:
        """Longest suffix of the history (at most N-1 tokens) that is a listed context."""
        h = tuple(int(t) for t in history)
        for j in range(min(len(h), self.N - 1), 0, -1):
            if self.is_context(h[len(h) - j:]):
                return h[len(h) - j:]
        return ()
