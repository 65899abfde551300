"""Speculation on/off by effective batch size (host logic).

The paper switches speculative decoding on under low load and off under high
load, using the runtime effective batch size as the load indicator and
thresholds found empirically per workload and hardware (Introduction; System
Design, "SuffixDecoding": adaptive enabling and disabling; Evaluation, the
decode-throughput-versus-batch-size figure).  This module holds that decision:
given measured verify-step times T(B, k) on this GPU (``bench.py --sweep``
produces them) and an acceptance model, it picks the draft length k (0 = plain
decode) that maximises accepted tokens per second at a batch size.

The switch itself needs no state: a verify step with k_max = 0 and one with
k_max > 0 take the same inputs (committed lengths and the pending token), so
consecutive steps may use different k.

Acceptance model: each draft token is accepted with probability ``alpha``
independently and acceptance stops at the first rejection, so a step with k
drafts emits  E[a + 1] = sum_{j=0..k} alpha^j  tokens on average.
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, Optional, Tuple


def expected_tokens(k: int, alpha: float) -> float:
    """Mean tokens emitted by one verify step with k drafts (the bonus position included)."""
    if k < 0 or not 0.0 <= alpha <= 1.0:
        raise ValueError("k >= 0 and 0 <= alpha <= 1")
    return float(sum(alpha ** j for j in range(k + 1)))


class SpecPolicy:
    """Draft-length choice from a table of measured step times.

    ``step_ms[(B, k)]`` is the time of one verify step (plus commit) for a batch
    of B requests with k drafts each.  Times at batch sizes between measured
    ones are interpolated linearly in log(B); outside the measured range the
    nearest measured batch size is used.
    """

    def __init__(self, step_ms: Dict[Tuple[int, int], float]):
        if not step_ms:
            raise ValueError("empty table")
        self.step_ms = dict(step_ms)
        self.ks = sorted({k for _, k in self.step_ms})
        self.batches = sorted({b for b, _ in self.step_ms})
        for b in self.batches:
            for k in self.ks:
                if (b, k) not in self.step_ms:
                    raise ValueError(f"table misses (B={b}, k={k})")

    def time_ms(self, batch: float, k: int) -> float:
        bs = self.batches
        if batch <= bs[0]:
            return self.step_ms[(bs[0], k)]
        if batch >= bs[-1]:
            return self.step_ms[(bs[-1], k)]
        for lo, hi in zip(bs, bs[1:]):
            if lo <= batch <= hi:
                t = (math.log(batch) - math.log(lo)) / (math.log(hi) - math.log(lo))
                return (1 - t) * self.step_ms[(lo, k)] + t * self.step_ms[(hi, k)]
        raise AssertionError("unreachable")

    def throughput(self, batch: float, k: int, alpha: float) -> float:
        """Modelled accepted tokens per second."""
        return batch * expected_tokens(k, alpha) / (self.time_ms(batch, k) * 1e-3)

    def choose_k(self, batch: float, alpha: float, ks: Optional[Iterable[int]] = None) -> int:
        """The k with the highest modelled throughput (ties -> the smaller k)."""
        best_k, best = None, -1.0
        for k in sorted(ks if ks is not None else self.ks):
            v = self.throughput(batch, k, alpha)
            if v > best * (1 + 1e-12):
                best_k, best = k, v
        return int(best_k)

    def crossover(self, alpha: float) -> Optional[float]:
        """Largest measured batch size at which some k > 0 still beats plain
        decode (None if speculation never wins)."""
        wins = [b for b in self.batches if self.choose_k(b, alpha) > 0]
        return float(max(wins)) if wins else None
