"""Oracle of the code-cache locality score and residency (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU baseline use
this module; the library never does.

The score of function f (Sec. 4.1, Eq. 3):

    l(f) = (1 - l_curr(f)) * (alpha * l_freq(f) + beta * sum_j l_asso(j | f)
                              + gamma * l_sema(f)) + l_curr(f)

with the components of App. B.1 (Eq. 8-10):

    l_freq(f)     = count(f) / max_j count(j)
    l_asso(j | f) = cooccur(f, j) / count(f)
    l_sema(f)     = PPL(f) / max_j PPL(j)

Readings where the paper leaves a choice:
  - the statistics cover the last ``window`` execution traces (one trace per
    task, the paper's trace length 20);
  - cooccur(f, j) counts the invocations of j that immediately follow an
    invocation of f within one trace (so sum_j l_asso(j | f) is the share of
    f's invocations that another call follows, within [0, 1]);
  - l_curr(f) = 1 iff f occurs in the most recent trace;
  - a component whose denominator is 0 is 0; PPL values are supplied by the
    caller (the language model that would measure them is out of scope);
  - residency (Alg. 1, the update step): functions in descending score, ties
    by ascending id, are kept on the GPU while their summed cost fits the
    budget; a function that does not fit is skipped and later ones are still
    considered;
  - the perplexity-based eviction threshold tau of the hyperparameter table
    (App. B.2, 15.0): functions whose perplexity is below tau -- code the model
    already predicts well, where the semantic term gives the least -- leave the
    GPU first.  Functions at or above tau are placed first (in score order),
    then the others (in score order) in what remains; tau = 0 leaves the plain
    score order;
  - entries that must stay on the GPU (read in place by a cache) are kept
    before anything else and their cost is counted first.
"""
from __future__ import annotations

from typing import List, Sequence

import numpy as np


class Locality:
    def __init__(self, n_funcs: int, window: int = 20, alpha: float = 0.4, beta: float = 0.3,
                 gamma: float = 0.3):
        if n_funcs < 1 or window < 1:
            raise ValueError("n_funcs and window must be >= 1")
        self.n = int(n_funcs)
        self.window = int(window)
        self.alpha, self.beta, self.gamma = float(alpha), float(beta), float(gamma)
        self.traces: List[List[int]] = []
        self.ppl = np.zeros(self.n)

    def record(self, trace: Sequence[int]) -> None:
        """One task's execution trace (function ids in call order)."""
        t = [int(f) for f in trace]
        if any(not (0 <= f < self.n) for f in t):
            raise ValueError("function id out of range")
        self.traces.append(t)
        if len(self.traces) > self.window:
            self.traces.pop(0)

    def set_ppl(self, f: int, ppl: float) -> None:
        if ppl < 0:
            raise ValueError("perplexity must be >= 0")
        self.ppl[int(f)] = float(ppl)

    # -- components ------------------------------------------------------------
    def counts(self) -> np.ndarray:
        c = np.zeros(self.n, dtype=np.int64)
        for t in self.traces:
            for f in t:
                c[f] += 1
        return c

    def cooccur(self) -> np.ndarray:
        """[f][j]: invocations of j immediately after f within one trace."""
        m = np.zeros((self.n, self.n), dtype=np.int64)
        for t in self.traces:
            for a, b in zip(t[:-1], t[1:]):
                m[a, b] += 1
        return m

    def l_freq(self) -> np.ndarray:
        c = self.counts()
        top = c.max()
        return c / top if top > 0 else np.zeros(self.n)

    def l_asso_sum(self) -> np.ndarray:
        c = self.counts()
        m = self.cooccur()
        out = np.zeros(self.n)
        for f in range(self.n):
            if c[f] > 0:
                out[f] = sum(m[f, j] / c[f] for j in range(self.n))
        return out

    def l_sema(self) -> np.ndarray:
        top = self.ppl.max()
        return self.ppl / top if top > 0 else np.zeros(self.n)

    def l_curr(self) -> np.ndarray:
        cur = np.zeros(self.n)
        if self.traces:
            for f in self.traces[-1]:
                cur[f] = 1.0
        return cur

    def scores(self) -> np.ndarray:
        freq, asso, sema, cur = self.l_freq(), self.l_asso_sum(), self.l_sema(), self.l_curr()
        out = np.empty(self.n)
        for f in range(self.n):
            mix = self.alpha * freq[f] + self.beta * asso[f] + self.gamma * sema[f]
            out[f] = (1.0 - cur[f]) * mix + cur[f]
        return out

    def residency(self, budget: int, cost: Sequence[int], tau: float = 0.0, pinned=None) -> np.ndarray:
        s = self.scores()
        keep = np.zeros(self.n, dtype=np.uint8)
        used = 0
        pinned = np.zeros(self.n, dtype=bool) if pinned is None else np.asarray(pinned, dtype=bool)
        for f in range(self.n):
            if pinned[f]:
                keep[f] = 1
                used += int(cost[f])
        order = sorted(range(self.n), key=lambda f: (-s[f], f))
        groups = [[f for f in order if self.ppl[f] >= tau], [f for f in order if self.ppl[f] < tau]] \
            if tau > 0 else [order]
        for group in groups:
            for f in group:
                if not keep[f] and used + int(cost[f]) <= budget:
                    keep[f] = 1
                    used += int(cost[f])
        return keep
