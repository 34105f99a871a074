"""Closed, normalised-by-construction synthetic n-gram models.

Model recipe (all randomness from one ``numpy.random.Generator``):

* Tokens ``0..V-1`` get Zipf ranks through a seeded permutation; the unigram
  distribution is Zipf(s) over the ranks.  If fewer than ``V`` unigrams are
  listed, the listed ones are the most frequent ranks and the others share one
  ``<unk>`` log-probability (the paper's start state stores every token, absent
  ones with the ``<unk>`` weight -- Section 2.2).
* Order ``k >= 2`` n-grams are drawn from the candidates ``(c, v)`` where ``c``
  is a listed order-(k-1) n-gram and ``c[1:] + (v,)`` is listed too.  That gives
  suffix closure, and prefix closure holds because ``c`` is listed.  Candidates
  are drawn without replacement with probability proportional to
  ``P(c) * P(v | c[1:])`` (successive sampling: exponential clocks when the
  candidate set is materialised, i.i.d. draws kept in first-seen order when it
  is too large to materialise).  Optional phrases force all their
  substrings of length <= N in first.
* For every context ``c`` with explicit continuations ``E(c)``: an explicit
  mass ``m_c ~ U(0.5, 0.95)`` (``1`` when ``E(c)`` covers the vocabulary) is
  split over ``E(c)`` in proportion to ``P(v | c[1:]) * exp(N(0, 1))``.  With
  ``l_c = sum_{v in E(c)} P(v | c[1:])`` (every term explicit by suffix
  closure) and ``Z(c[1:])`` the total mass of the shorter context as stored,
  the backoff weight ``B(c) = ln(1 - m_c) - ln(Z(c[1:]) - l_c)`` makes
  ``sum_v P(v | c) = 1`` under the backoff rule W(t|c) = B(c) + W(t|c[1:])
  (Section 2.1).  Weights are rounded to fp32 first and the backoff is computed
  from the rounded values and the stored mass Z of the shorter context (not
  from an assumed 1: when ``1 - l_c`` is small, the rounding residue of the
  shorter context would otherwise be amplified by ``1 / (1 - l_c)``), so the
  stored model is normalised to ~1e-7 at every depth.

All weights are natural logarithms.  The model is kept per order as a trie
level: ``pid`` (row of the prefix in the order below), ``tok`` (last token),
``sid`` (row of the suffix in the order below), rows sorted by ``(pid, tok)``,
which is lexicographic order of the token tuples.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

# Largest candidate set that is materialised for exact exponential-clock
# sampling; beyond it candidates are drawn i.i.d. and deduplicated.
_MATERIALISE_LIMIT = 40_000_000


@dataclass
class Level:
    pid: np.ndarray   # int64 [n]  row of prefix in level k-1 (level 0: root row 0)
    tok: np.ndarray   # int32 [n]  last token
    sid: np.ndarray   # int64 [n]  row of suffix in level k-1
    W: np.ndarray     # float32 [n] log P(tok | prefix), nats
    B: np.ndarray     # float32 [n] backoff weight of the n-gram as a context
    cum: np.ndarray   # float64 [n] log-probability of the n-gram as a sequence


@dataclass
class NgramModel:
    vocab_size: int
    max_order: int
    levels: List[Level]               # levels[0] is the root placeholder
    unk_logprob: float = float("nan")
    phrases: Optional[List[np.ndarray]] = None
    bos_eos: bool = False             # token V is <s> (context only), V + 1 is </s> (predicted only)
    _tokens_cache: dict = field(default_factory=dict, repr=False)

    @property
    def bos(self) -> int:
        return self.vocab_size

    @property
    def eos(self) -> int:
        return self.vocab_size + 1

    def is_state_row(self, k: int) -> np.ndarray:
        """Rows of level k that are contexts (all of them, except n-grams ending in </s>)."""
        tok = self.levels[k].tok
        return tok != self.eos if self.bos_eos else np.ones(len(tok), bool)

    @property
    def counts(self) -> List[int]:
        return [len(l.tok) for l in self.levels[1:]]

    @property
    def num_ngrams(self) -> int:
        return int(sum(self.counts))

    @property
    def num_states(self) -> int:
        """Root plus every listed context of order < N (the highest order has no states)."""
        return 1 + int(sum(int(self.is_state_row(k).sum()) for k in range(1, self.max_order)))

    def state_offset(self, k: int) -> int:
        """Canonical id of the first order-k state (k < N): root 0, then by order, then lexicographic."""
        assert 1 <= k < self.max_order
        return 1 + int(sum(int(self.is_state_row(j).sum()) for j in range(1, k)))

    @property
    def start_state(self) -> int:
        """State of the context <s> (bos_eos models), else the empty context."""
        if not self.bos_eos or self.max_order < 2:
            return 0
        return int(state_ids_of(self, np.array([[self.bos]]))[0])

    def level_tokens(self, k: int) -> np.ndarray:
        """[n_k, k] int32 token tuples of level k, in lexicographic order."""
        if k in self._tokens_cache:
            return self._tokens_cache[k]
        lv = self.levels[k]
        if k == 1:
            t = lv.tok.astype(np.int32)[:, None]
        else:
            prev = self.level_tokens(k - 1)
            t = np.concatenate([prev[lv.pid], lv.tok[:, None].astype(np.int32)], axis=1)
        self._tokens_cache[k] = t
        return t

    def to_list(self, shuffle_seed: Optional[int] = None):
        """Return the n-gram list as ``(order, tokens, logprob, backoff)`` arrays.

        ``tokens`` is ``[M, N]`` int32; row i uses its first ``order[i]`` entries
        (context first, predicted token last) and is padded with -1.  Rows are in
        canonical order unless ``shuffle_seed`` is given.
        """
        N = self.max_order
        M = self.num_ngrams
        order = np.empty(M, np.int32)
        tokens = np.full((M, N), -1, np.int32)
        logprob = np.empty(M, np.float32)
        backoff = np.empty(M, np.float32)
        o = 0
        for k in range(1, N + 1):
            lv = self.levels[k]
            n = len(lv.tok)
            order[o:o + n] = k
            tokens[o:o + n, :k] = self.level_tokens(k)
            logprob[o:o + n] = lv.W
            backoff[o:o + n] = lv.B
            o += n
        if shuffle_seed is not None:
            p = np.random.default_rng(shuffle_seed).permutation(M)
            order, tokens, logprob, backoff = order[p], tokens[p], logprob[p], backoff[p]
        return (np.ascontiguousarray(order), np.ascontiguousarray(tokens),
                np.ascontiguousarray(logprob), np.ascontiguousarray(backoff))


def lookup_ids(model: NgramModel, tuples: np.ndarray) -> np.ndarray:
    """Row index, within its level, of each token tuple ([n, k] int); -1 if not listed."""
    tuples = np.asarray(tuples, dtype=np.int64)
    n, k = tuples.shape
    V = model.vocab_size
    lv1 = model.levels[1]
    pos = np.searchsorted(lv1.tok, tuples[:, 0])
    pos = np.minimum(pos, len(lv1.tok) - 1)
    ok = lv1.tok[pos] == tuples[:, 0]
    ids = np.where(ok, pos, -1)
    for j in range(2, k + 1):
        lv = model.levels[j]
        key = lv.pid * V + lv.tok
        q = ids * V + tuples[:, j - 1]
        p = np.searchsorted(key, q)
        p = np.minimum(p, len(key) - 1)
        ok = (ids >= 0) & (key[p] == q)
        ids = np.where(ok, p, -1)
    return ids


def state_ids_of(model: NgramModel, tuples: np.ndarray) -> np.ndarray:
    """Canonical state ids of context tuples ([n, k] with 1 <= k < N); -1 if not a state."""
    tuples = np.asarray(tuples)
    k = tuples.shape[1]
    rows = lookup_ids(model, tuples)
    ok = model.is_state_row(k)
    rank = np.cumsum(ok) - 1                     # rank among the level's contexts
    ids = np.where(rows >= 0, rank[np.maximum(rows, 0)] + model.state_offset(k), -1)
    ids = np.where((rows >= 0) & ok[np.maximum(rows, 0)], ids, -1)
    return ids.astype(np.int32)


def _zipf_unigrams(V: int, n1: int, s: float, rng: np.random.Generator):
    perm = rng.permutation(V)                     # perm[r] = token of Zipf rank r
    zipf = 1.0 / np.arange(1, V + 1, dtype=np.float64) ** s
    zipf /= zipf.sum()
    if n1 == V:
        p = np.empty(V)
        p[perm] = zipf
        return np.arange(V, dtype=np.int32), p, float("nan")
    if not 1 <= n1 < V:
        raise ValueError("unigram count must be in [1, V]")
    listed = np.sort(perm[:n1]).astype(np.int32)
    p_unk = float(zipf[n1:].mean())
    unk32 = np.float32(np.log(p_unk))
    mass = 1.0 - (V - n1) * float(np.exp(np.float64(unk32)))
    p_all = np.empty(V)
    p_all[perm] = zipf
    p = p_all[listed]
    p = p * (mass / p.sum())
    return listed, p, float(unk32)


def _select_candidates(prev: Level, grand_n: int, need: int, forced: np.ndarray,
                       rng: np.random.Generator, ctx_ok: Optional[np.ndarray] = None,
                       cand_ok: Optional[np.ndarray] = None) -> np.ndarray:
    """Keys ``c * n_prev + y`` of the chosen order-k n-grams (c: prefix row, y: suffix row).

    ``ctx_ok`` marks the rows that may be extended (contexts), ``cand_ok`` the
    rows whose last token may be appended (predictable tokens)."""
    n_prev = len(prev.tok)
    nodes = np.arange(grand_n)
    cb = np.searchsorted(prev.pid, nodes, "left")
    ce = np.searchsorted(prev.pid, nodes, "right")
    s = prev.sid
    lens = (ce - cb)[s]
    if ctx_ok is not None:
        lens = np.where(ctx_ok, lens, 0)
    forced = np.unique(forced.astype(np.int64))
    if len(forced) > need:
        raise ValueError("more forced n-grams than the order's count")
    masked = cand_ok is not None and not cand_ok.all()
    total = int(lens.sum())
    if masked or total <= _MATERIALISE_LIMIT:
        c_idx = np.repeat(np.arange(n_prev, dtype=np.int64), lens)
        starts = np.repeat(cb[s], lens)
        offs = np.arange(total, dtype=np.int64) - np.repeat(np.cumsum(lens) - lens, lens)
        y = starts + offs
        del starts, offs
        if masked:
            keep = cand_ok[y]
            c_idx, y = c_idx[keep], y[keep]
            total = len(y)
        if total <= need:
            return np.sort(c_idx * n_prev + y)
        keys = c_idx * n_prev + y
        # exponential clocks: smaller log(E) - log w is drawn earlier
        score = np.log(rng.exponential(size=total)) - (prev.cum[c_idx] + prev.W[y].astype(np.float64))
        del c_idx, y
        if len(forced):
            score[np.isin(keys, forced)] = -np.inf
        take = np.argpartition(score, need - 1)[:need]
        return np.sort(keys[take])
    # i.i.d. draws proportional to P(c) * P(v | c[1:]), first-seen distinct keys kept
    ew = np.exp(prev.W.astype(np.float64))
    cumew = np.concatenate([[0.0], np.cumsum(ew)])
    mass = cumew[ce] - cumew[cb]
    wc = np.exp(prev.cum - prev.cum.max()) * mass[s]
    if ctx_ok is not None:
        wc = wc * ctx_ok
    cdf = np.cumsum(wc)
    cdf /= cdf[-1]
    chosen = [forced]
    seen = forced                      # sorted distinct keys drawn so far
    have = len(forced)
    batch = int(1.5 * (need - have)) + 1024
    for _ in range(256):
        # sorted queries keep the binary searches cache-friendly; the draws are
        # shuffled afterwards so their order is that of i.i.d. draws again
        c = np.searchsorted(cdf, np.sort(rng.random(batch)), "right")
        c = np.minimum(c, n_prev - 1)
        sc = s[c]
        lo_i, hi_i = cb[sc], ce[sc]
        u = cumew[lo_i] + rng.random(batch) * (cumew[hi_i] - cumew[lo_i])
        ou = np.argsort(u)
        y = np.empty(batch, np.int64)
        y[ou] = np.searchsorted(cumew, u[ou], "right") - 1
        y = np.clip(y, lo_i, hi_i - 1)
        draws = c.astype(np.int64) * n_prev + y
        draws = draws[rng.permutation(batch)]
        uniq, first = np.unique(draws, return_index=True)
        if len(seen):
            p = np.minimum(np.searchsorted(seen, uniq), len(seen) - 1)
            fresh = seen[p] != uniq
            uniq, first = uniq[fresh], first[fresh]
        new = uniq[np.argsort(first, kind="stable")][: need - have]
        chosen.append(new)
        have += len(new)
        if have >= need:
            return np.sort(np.concatenate(chosen))
        seen = np.sort(np.concatenate([seen, new]))
        batch = max(int(4.0 * (need - have)), 1 << 21)
    raise RuntimeError("candidate sampling did not reach the requested count")


def _assign_probabilities(prev: Level, pid: np.ndarray, sid: np.ndarray, n_pred: int,
                          z_low: np.ndarray, rng: np.random.Generator):
    """Weights of the new level; backoff weights and stored mass Z of its contexts.

    ``z_low[c]`` is the stored mass of context c's suffix c[1:].  Sets
    ``prev.B`` and returns ``(W, Z)`` with Z the stored mass of each context of
    the previous level under the backoff rule.
    """
    n_prev = len(prev.tok)
    p_low = np.exp(prev.W[sid].astype(np.float64))        # explicit by suffix closure
    raw = p_low * np.exp(rng.standard_normal(len(pid)))
    gsum = np.bincount(pid, weights=raw, minlength=n_prev)
    l = np.bincount(pid, weights=p_low, minlength=n_prev)
    cnt = np.bincount(pid, minlength=n_prev)
    m = rng.uniform(0.5, 0.95, size=n_prev)
    full = cnt == n_pred          # every predictable token continues the context
    m[full] = 1.0
    P = m[pid] * raw / gsum[pid]
    W = np.log(P).astype(np.float32)
    m32 = np.bincount(pid, weights=np.exp(W.astype(np.float64)), minlength=n_prev)
    B = np.zeros(n_prev)
    has = (cnt > 0) & ~full
    compl = np.maximum(z_low[has] - l[has], 1e-12)        # mass left to the backoff
    B[has] = np.log1p(-np.minimum(m32[has], 1.0 - 1e-12)) - np.log(compl)
    prev.B = B.astype(np.float32)
    Z = z_low.copy()                                       # no continuations: all mass backs off
    Z[full] = m32[full]
    Z[has] = m32[has] + np.exp(prev.B[has].astype(np.float64)) * compl
    return W, Z


# The <s> unigram is a context only; its weight (log10 -99 as KenLM writes it)
# is never scored.
BOS_LOGPROB = float(np.float32(-99.0 * np.log(10.0)))


def generate_model(V: int, counts: Sequence[int], zipf_s: float, seed: int,
                   phrases: Optional[Sequence[Sequence[int]]] = None, bos_eos: bool = False,
                   eos_prob: float = 0.04) -> NgramModel:
    """Generate a closed, normalised n-gram model with ``counts[k-1]`` n-grams of order k.

    With ``bos_eos``, token V is ``<s>`` (it opens contexts and is never
    predicted) and V + 1 is ``</s>`` (it is predicted with unigram probability
    ``eos_prob`` and never extended); every context then sums to one over the V
    tokens and ``</s>``.  counts[0] counts the unigrams of the V tokens only.
    """
    N = len(counts)
    if N < 1:
        raise ValueError("need at least one order")
    rng = np.random.default_rng(seed)
    root = Level(pid=np.zeros(1, np.int64), tok=np.zeros(1, np.int32), sid=np.zeros(1, np.int64),
                 W=np.zeros(1, np.float32), B=np.zeros(1, np.float32), cum=np.zeros(1))
    toks, p1, unk = _zipf_unigrams(V, int(counts[0]), zipf_s, rng)
    n_pred = V
    if bos_eos:
        if not np.isnan(unk):
            raise ValueError("bos_eos models list every token")
        p1 = p1 * (1.0 - eos_prob)
        toks = np.concatenate([toks, [V, V + 1]]).astype(np.int32)
        W1 = np.concatenate([np.log(p1), [BOS_LOGPROB, np.log(eos_prob)]]).astype(np.float32)
        n_pred = V + 1
    else:
        W1 = np.log(p1).astype(np.float32)
    lv1 = Level(pid=np.zeros(len(toks), np.int64), tok=toks, sid=np.zeros(len(toks), np.int64),
                W=W1, B=np.zeros(len(toks), np.float32), cum=W1.astype(np.float64))
    model = NgramModel(vocab_size=V, max_order=N, levels=[root, lv1], unk_logprob=unk,
                       phrases=[np.asarray(p, np.int64) for p in phrases] if phrases is not None else None,
                       bos_eos=bos_eos)
    pred1 = toks != V if bos_eos else np.ones(len(toks), bool)
    if bos_eos:
        lv1.cum = np.where(pred1, lv1.cum, np.log(0.05))   # <s> opens contexts as often as a frequent word
    z_root = float(np.exp(W1.astype(np.float64))[pred1].sum())
    if not np.isnan(unk):
        z_root += (V - len(toks)) * float(np.exp(np.float64(np.float32(unk))))
    z_levels = [np.array([z_root])]                        # Z per context, level by level
    for k in range(2, N + 1):
        prev = model.levels[k - 1]
        grand_n = len(model.levels[k - 2].tok)
        n_prev = len(prev.tok)
        forced = np.zeros(0, np.int64)
        if model.phrases:
            subs = [p[i:i + k] for p in model.phrases for i in range(len(p) - k + 1)]
            if subs:
                subs = np.unique(np.stack(subs), axis=0)
                c = lookup_ids(model, subs[:, :-1])
                y = lookup_ids(model, subs[:, 1:])
                if (c < 0).any() or (y < 0).any():
                    raise ValueError("phrase tokens must all be listed unigrams")
                forced = c * n_prev + y
        ctx_ok = cand_ok = None
        if bos_eos:
            ctx_ok = prev.tok != V + 1                     # </s> ends a sentence: no context
            cand_ok = prev.tok != V                        # <s> is never predicted
        keys = _select_candidates(prev, grand_n, int(counts[k - 1]), forced, rng, ctx_ok, cand_ok)
        pid = keys // n_prev
        sid = keys % n_prev
        tok = prev.tok[sid]
        order = np.lexsort((tok, pid))
        pid, sid, tok = pid[order], sid[order], tok[order]
        # stored mass of each context's suffix: Z of the level below (the root for unigrams)
        z_low = z_levels[k - 2][prev.sid]
        W, z_prev = _assign_probabilities(prev, pid, sid, n_pred, z_low, rng)
        z_levels.append(z_prev)
        cum = prev.cum[pid] + W.astype(np.float64)
        model.levels.append(Level(pid=pid, tok=tok.astype(np.int32), sid=sid, W=W,
                                  B=np.zeros(len(tok), np.float32), cum=cum))
    return model
