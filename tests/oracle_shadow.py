"""Independent set-semantics bookkeeping used to pin the oracle.

Nothing here looks at the retrospective mask A or the kernel mask M: it keeps
the history of selected page sets and token positions and derives, straight
from eq. (update-sup), which pages a past query may still attend:

    eligible(t, tau) = S_t  minus  (S_tau u ... u S_{t-1})
                       minus  { p : p holds a key newer than tau's query }

(the last term is the causality rule that Alg. 2's current-page rule enforces), and,
for brute force, the set of token positions each query has attended so far.
"""
from __future__ import annotations

from typing import Dict, List, Set

import numpy as np


class Shadow:
    def __init__(self, batch: int, num_kv_heads: int, page_size: int, window: int):
        self.batch, self.hk, self.P, self.W = batch, num_kv_heads, page_size, window
        self.S: Dict[int, List[List[Set[int]]]] = {}   # step -> [b][h] -> selected set
        self.qpos: Dict[int, List[int]] = {}            # step -> [b] -> query position
        # (b, h, tau) -> set of attended token positions
        self.seen: Dict[tuple, Set[int]] = {}

    def eligible(self, t: int, b: int, h: int, tau: int, seq_len: int) -> Set[int]:
        S_t = self.S[t][b][h]
        union: Set[int] = set()
        for m in range(tau, t):
            union |= self.S[m][b][h]
        out = set()
        for p in S_t - union:
            last = min((p + 1) * self.P, seq_len) - 1
            if last <= self.qpos[tau][b]:
                out.add(p)
        return out

    def record(self, t: int, selected: np.ndarray, num: np.ndarray, seq_lens: np.ndarray):
        """Record step t's selection; returns {(b,h,tau): eligible page set} for its
        past queries and the current one (the current query sees all of S_t)."""
        self.S[t] = [[set(int(p) for p in selected[b, h, :num[b, h]]) for h in range(self.hk)]
                     for b in range(self.batch)]
        self.qpos[t] = [int(seq_lens[b]) - 1 for b in range(self.batch)]
        res = {}
        for b in range(self.batch):
            L = int(seq_lens[b])
            for h in range(self.hk):
                for tau in range(max(0, t - self.W), t + 1):
                    if tau == t:
                        pages = set(self.S[t][b][h])
                    else:
                        pages = self.eligible(t, b, h, tau, L)
                    res[(b, h, tau)] = pages
                    toks = set()
                    for p in pages:
                        toks.update(range(p * self.P, min((p + 1) * self.P, L)))
                    key = (b, h, tau)
                    prev = self.seen.setdefault(key, set())
                    assert not (prev & toks), "a token would be counted twice"
                    prev |= toks
        return res


def softmax_attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, toks, scale: float):
    """Brute-force fp64 softmax attention of one query over a token set."""
    toks = sorted(toks)
    if not toks:
        return np.zeros(V.shape[-1]), -np.inf
    k = K[toks].astype(np.float64)
    v = V[toks].astype(np.float64)
    s = scale * (k @ q.astype(np.float64))
    m = s.max()
    w = np.exp(s - m)
    return (w @ v) / w.sum(), m + np.log(w.sum())
