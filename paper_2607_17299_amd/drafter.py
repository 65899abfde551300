"""Host-side suffix-match drafter (model-free speculation), test-harness logic.

SuffixDecoding keeps the token sequences of earlier trajectories and, while a
request decodes, matches the end of its current context against them to
propose the tokens that followed (System Design, "SuffixDecoding").  WAR keeps
it on the host, lets outside code add finished trajectories (its "external
update interface"), and after each RL step broadcasts every trajectory to all
workers so that all of them draft from the same history.

This drafter proposes a chain (no speculation tree):
  1. take the last ``max_match`` tokens of the context as the pattern;
  2. find the longest suffix of the pattern that occurs in the stored
     trajectories and is followed by at least one token;
  3. among the tokens that follow its occurrences pick the most frequent
     (ties -> the token whose first such occurrence comes earliest);
  4. append it to the pattern and repeat until k tokens are drafted or no
     suffix of length >= 1 matches.
Trajectories are stored back to back with a separator that never matches, so
no match crosses a trajectory boundary.  Draft tokens are inputs of the verify
step; this module holds none of its arithmetic.
"""
from __future__ import annotations

from typing import List, Sequence

import numpy as np

_SEP = -1


class SuffixDrafter:
    def __init__(self, max_match: int = 64):
        self.max_match = max_match
        self._parts: List[np.ndarray] = []
        self._corpus = np.full(1, _SEP, dtype=np.int64)
        self._dirty = False

    def add_trajectory(self, tokens: Sequence[int]) -> None:
        """External update interface: add one finished trajectory."""
        self._parts.append(np.asarray(tokens, dtype=np.int64))
        self._dirty = True

    def _build(self) -> None:
        if self._dirty:
            pieces = [np.full(1, _SEP, np.int64)]
            for p in self._parts:
                pieces += [p, np.full(1, _SEP, np.int64)]
            self._corpus = np.concatenate(pieces)
            self._dirty = False

    def _longest_match(self, pattern: np.ndarray) -> np.ndarray:
        """End positions (in the corpus) of the longest matching suffix, or empty."""
        c = self._corpus
        if len(pattern) == 0:
            return np.zeros(0, np.int64)
        cand = np.nonzero(c[:-1] == pattern[-1])[0]     # must be followed by a position
        cand = cand[c[cand + 1] != _SEP]
        best = cand
        L = 1
        while len(cand) and L < len(pattern):
            prev = cand - L
            ok = prev >= 0
            cand = cand[ok]
            cand = cand[c[cand - L] == pattern[-1 - L]]
            if len(cand) == 0:
                break
            best = cand
            L += 1
        return best

    def propose(self, context: Sequence[int], k: int) -> List[int]:
        self._build()
        pat = list(np.asarray(context, dtype=np.int64)[-self.max_match:])
        out: List[int] = []
        for _ in range(k):
            ends = self._longest_match(np.asarray(pat[-self.max_match:], dtype=np.int64))
            if len(ends) == 0:
                break
            nxt = self._corpus[ends + 1]
            toks, first, counts = np.unique(nxt, return_index=True, return_counts=True)
            best = np.lexsort((first, -counts))[0]     # most frequent, then earliest
            t = int(toks[best])
            out.append(t)
            pat.append(t)
        return out


def brute_force_propose(trajectories: Sequence[Sequence[int]], context: Sequence[int], k: int,
                        max_match: int = 64) -> List[int]:
    """Pure-Python scan with the same definition (used to pin SuffixDrafter)."""
    corpus: List[int] = [_SEP]
    for t in trajectories:
        corpus += [int(x) for x in t] + [_SEP]
    pat = [int(x) for x in context][-max_match:]
    out: List[int] = []
    for _ in range(k):
        p = pat[-max_match:]
        best_len, best_ends = 0, []
        for e in range(len(corpus) - 1):
            if corpus[e + 1] == _SEP:
                continue
            L = 0
            while L < len(p) and e - L >= 0 and corpus[e - L] == p[-1 - L]:
                L += 1
            if L > best_len:
                best_len, best_ends = L, [e]
            elif L == best_len and L > 0:
                best_ends.append(e)
        if best_len == 0:
            break
        counts, first = {}, {}
        for i, e in enumerate(best_ends):
            t = corpus[e + 1]
            counts[t] = counts.get(t, 0) + 1
            first.setdefault(t, i)
        t = min(counts, key=lambda x: (-counts[x], first[x]))
        out.append(t)
        pat.append(t)
    return out
