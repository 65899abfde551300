"""Host-side suffix-match drafter (model-free speculation), test-harness logic.

SuffixDecoding keeps the token sequences of earlier trajectories and, while a
request decodes, matches the end of its current context against them to
propose the tokens that followed (System Design, "SuffixDecoding").  WAR keeps
it on the host, lets outside code add finished trajectories (its "external
update interface"), and after each RL step broadcasts every trajectory to all
workers so that all of them draft from the same history.

``propose`` drafts a chain:
  1. take the last ``max_match`` tokens of the context as the pattern;
  2. find the longest suffix of the pattern that occurs in the stored
     trajectories and is followed by at least one token;
  3. among the tokens that follow its occurrences pick the most frequent
     (ties -> the token whose first such occurrence comes earliest);
  4. append it to the pattern and repeat until k tokens are drafted or no
     suffix of length >= 1 matches.
``propose_tree`` drafts a speculation tree of at most n nodes (SuffixDecoding
grows its trees by the empirical frequencies of the stored continuations).
Reading: best-first growth.  A candidate child of a node is a token that
follows the node's longest matching suffix, scored by the node's score times
the token's share of those continuations (the root scores 1).  The best
candidate (ties -> the one proposed first; a node's children are proposed
most frequent first, then by earliest occurrence) becomes the next node, and
its own children join the candidates.  Nodes are numbered in the order they
are taken, so every parent precedes its children.
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
        self._dirty = True

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
            # token -> its positions (ascending), every position but the last:
            # a stable sort groups equal tokens and keeps their order
            head = self._corpus[:-1]
            self._pos = np.argsort(head, kind="stable")
            self._vals, self._start = np.unique(head[self._pos], return_index=True)
            self._dirty = False

    def _positions(self, tok: int) -> np.ndarray:
        """Ascending corpus positions (except the last) holding `tok`."""
        i = int(np.searchsorted(self._vals, tok))
        if i >= len(self._vals) or self._vals[i] != tok:
            return np.zeros(0, np.int64)
        end = self._start[i + 1] if i + 1 < len(self._vals) else len(self._pos)
        return self._pos[self._start[i]:end]

    def _longest_match(self, pattern: np.ndarray) -> np.ndarray:
        """End positions (in the corpus) of the longest matching suffix, or empty."""
        c = self._corpus
        if len(pattern) == 0:
            return np.zeros(0, np.int64)
        cand = self._positions(int(pattern[-1]))         # must be followed by a position
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

    def _continuations(self, pat: List[int]):
        """(token, count) after the longest matching suffix of pat, most frequent
        first, ties by earliest occurrence; and the number of occurrences."""
        ends = self._longest_match(np.asarray(pat[-self.max_match:], dtype=np.int64))
        if len(ends) == 0:
            return [], 0
        nxt = self._corpus[ends + 1]
        toks, first, counts = np.unique(nxt, return_index=True, return_counts=True)
        order = np.lexsort((first, -counts))
        return [(int(toks[i]), int(counts[i])) for i in order], len(ends)

    def propose_tree(self, context: Sequence[int], n: int):
        """Up to n draft nodes: (tokens, parents), parents[i] in [0, i] is the
        parent of node i + 1 (node 0 is the context's last token)."""
        self._build()
        base = [int(x) for x in np.asarray(context, dtype=np.int64)[-self.max_match:]]
        tokens: List[int] = []
        parents: List[int] = []
        paths = {0: []}
        cand = []          # (-score, proposal order, parent node, token)
        order = 0

        def expand(node: int, score: float):
            nonlocal order
            conts, total = self._continuations(base + paths[node])
            for t, c in conts[:n]:
                cand.append((-score * c / total, order, node, t))
                order += 1

        expand(0, 1.0)
        while cand and len(tokens) < n:
            cand.sort()
            neg, _, par, t = cand.pop(0)
            tokens.append(t)
            parents.append(par)
            j = len(tokens)
            paths[j] = paths[par] + [t]
            expand(j, -neg)
        return tokens, parents

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


def _brute_counts(corpus: List[int], p: List[int]):
    """Tokens after the longest matching suffix of p: counts, first occurrence
    rank, and the number of occurrences (pure-Python scan)."""
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
    counts, first = {}, {}
    if best_len == 0:
        return counts, first, 0
    for i, e in enumerate(best_ends):
        t = corpus[e + 1]
        counts[t] = counts.get(t, 0) + 1
        first.setdefault(t, i)
    return counts, first, len(best_ends)


def _brute_corpus(trajectories) -> List[int]:
    corpus: List[int] = [_SEP]
    for t in trajectories:
        corpus += [int(x) for x in t] + [_SEP]
    return corpus


def brute_force_propose(trajectories: Sequence[Sequence[int]], context: Sequence[int], k: int,
                        max_match: int = 64) -> List[int]:
    """Pure-Python scan with the same definition (used to pin SuffixDrafter)."""
    corpus = _brute_corpus(trajectories)
    pat = [int(x) for x in context][-max_match:]
    out: List[int] = []
    for _ in range(k):
        counts, first, _ = _brute_counts(corpus, pat[-max_match:])
        if not counts:
            break
        t = min(counts, key=lambda x: (-counts[x], first[x]))
        out.append(t)
        pat.append(t)
    return out


def brute_force_propose_tree(trajectories: Sequence[Sequence[int]], context: Sequence[int], n: int,
                             max_match: int = 64):
    """Best-first tree growth written as a plain scan: at every step, rescan all
    taken nodes' continuations and take the best one not yet taken."""
    corpus = _brute_corpus(trajectories)
    base = [int(x) for x in context][-max_match:]
    nodes = [([], 1.0, 0)]              # (path tokens, score, proposal rank)
    tokens: List[int] = []
    parents: List[int] = []
    rank = {}                           # (node, token) -> global proposal order
    seq = 0
    while len(tokens) < n:
        best = None
        for j, (path, score, _) in enumerate(nodes):
            counts, first, total = _brute_counts(corpus, (base + path)[-max_match:])
            ranked = sorted(counts, key=lambda x: (-counts[x], first[x]))[:n]
            for t in ranked:
                if (j, t) not in rank:
                    rank[(j, t)] = seq
                    seq += 1
                if any(parents[i] == j and tokens[i] == t for i in range(len(tokens))):
                    continue
                key = (-score * counts[t] / total, rank[(j, t)])
                if best is None or key < best[0]:
                    best = (key, j, t)
        if best is None:
            break
        (neg, _), j, t = best
        tokens.append(t)
        parents.append(j)
        nodes.append((nodes[j][0] + [t], -neg, 0))
    return tokens, parents
