"""ARPA text from a generated model (test input for the library's ARPA reader).

Writes base-10 logarithms (the natural-log weights divided by ln 10, printed
with 17 significant digits), one section per order, backoff weights on every
context line, <unk> when the model has an <unk> weight, and <s> / </s> for
models with sentence markers.
"""

from __future__ import annotations

import math
from typing import Sequence

import numpy as np

from .ngram import NgramModel

LN10 = math.log(10.0)


def write_arpa(model: NgramModel, vocab: Sequence[str]) -> str:
    V, N = model.vocab_size, model.max_order
    words = list(vocab) + (["<s>", "</s>"] if model.bos_eos else [])
    counts = list(model.counts)
    has_unk = not np.isnan(model.unk_logprob)
    if has_unk:
        counts[0] += 1
    out = ["", "\\data\\"]
    out += [f"ngram {k}={counts[k - 1]}" for k in range(1, N + 1)]
    for k in range(1, N + 1):
        out += ["", f"\\{k}-grams:"]
        lv = model.levels[k]
        toks = model.level_tokens(k)
        if k == 1 and has_unk:
            out.append(f"{float(model.unk_logprob) / LN10!r}\t<unk>\t0")
        eos_row = (lv.tok == V + 1) if model.bos_eos else np.zeros(len(lv.tok), bool)
        for i in range(len(lv.tok)):
            ctx = " ".join(words[t] for t in toks[i])
            line = f"{float(lv.W[i]) / LN10!r}\t{ctx}"
            if k < N and not eos_row[i]:
                line += f"\t{float(lv.B[i]) / LN10!r}"
            out.append(line)
    out += ["", "\\end\\", ""]
    return "\n".join(out)


def bpe_like_vocab(V: int):
    """V distinct word strings shaped like subword units."""
    return [f"▁w{i}" if i % 3 == 0 else f"t{i}" for i in range(V)]


def write_arpa_list(V: int, N: int, order, tokens, logprob, backoff, unk_logprob, vocab: Sequence[str],
                    bos_eos: bool = False) -> str:
    """ARPA text of an n-gram list in any order (natural-log weights), e.g. a
    pruned list that is not closed; rows are written per order as given."""
    words = list(vocab) + (["<s>", "</s>"] if bos_eos else [])
    order = np.asarray(order)
    has_unk = not np.isnan(unk_logprob)
    counts = [int((order == k).sum()) for k in range(1, N + 1)]
    if has_unk:
        counts[0] += 1
    out = ["", "\\data\\"]
    out += [f"ngram {k}={counts[k - 1]}" for k in range(1, N + 1)]
    for k in range(1, N + 1):
        out += ["", f"\\{k}-grams:"]
        if k == 1 and has_unk:
            out.append(f"{float(unk_logprob) / LN10!r}\t<unk>\t0")
        for i in np.flatnonzero(order == k):
            toks = [int(t) for t in tokens[i][:k]]
            line = f"{float(logprob[i]) / LN10!r}\t{' '.join(words[t] for t in toks)}"
            if k < N and not (bos_eos and toks[-1] == V + 1):
                line += f"\t{float(backoff[i]) / LN10!r}"
            out.append(line)
    out += ["", "\\end\\", ""]
    return "\n".join(out)
