"""Greedy verification of draft tokens -- oracle (test infrastructure only).

The paper requires speculative decoding to be lossless: the accepted output is
what the target model alone would emit (Introduction; Background, "Why Workload
Matters").  Its rollouts sample, but it states no verification rule; the
reading taken here is greedy decoding, for which losslessness means:

  row i of the block holds the token at position c+i (row 0 = the pending
  token, rows 1..n = drafts d_1..d_n);  g_i = argmax of row i's logits is the
  target's greedy choice for position c+i+1;  draft d_m is accepted iff every
  earlier draft was and d_m == g_{m-1};  the step emits the accepted drafts
  and then the target's own token g_a (the "bonus" token), a+1 tokens in all.

Argmax ties go to the lowest token id.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np


def argmax_lowest(z: np.ndarray) -> np.ndarray:
    """Per-row argmax of z [..., V]; among equal maxima the lowest index wins."""
    z = np.asarray(z)
    if np.isnan(z).any():
        raise ValueError("NaN logits")
    m = z.max(axis=-1, keepdims=True)
    return np.argmax(z == m, axis=-1)       # first True = lowest id at the max


def accept_length(drafts: Sequence[int], greedy: Sequence[int]) -> int:
    """Largest a <= len(drafts) with drafts[m] == greedy[m] for every m < a."""
    a = 0
    for d, g in zip(drafts, greedy):
        if int(d) != int(g):
            break
        a += 1
    return a


def top2_gap(z: np.ndarray) -> np.ndarray:
    """Difference between the largest and second-largest logit of each row."""
    s = np.sort(np.asarray(z, dtype=np.float64), axis=-1)
    return s[..., -1] - s[..., -2]
