"""Comparison rules shared by the GPU parity tests.

Floating point: logits within max-abs 5e-2 of the oracle (bf16 compute, fp32
accumulate against the float64 oracle with the same bf16 rounding points).
At full depth (36 layers) no fp32-accumulating implementation meets 5e-2:
the oracle's own fp32-accumulation mode drifts ~0.12 from its float64 mode on
the same inputs, because the rounding points amplify summation-order noise
layer after layer.  There the bound is max(5e-2, 1.5 x that measured drift),
computed in the test from the oracle alone (fp32_drift_tol).

Integers decided by floating point (greedy tokens, accept lengths, next
tokens): bit-exact, except where the oracle's top-2 logit gap is below 0.1
(a near-tie), which is reported instead of failed.  A mismatch at a row whose
oracle gap exceeds twice the row's measured max |logit error| is always a
failure: with every logit within half the gap, the argmax cannot change.
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np

from oracle.accept import argmax_lowest, top2_gap

LOGIT_TOL = 5e-2
NEAR_TIE = 0.1


def fp32_drift_tol(o64: np.ndarray, o32: np.ndarray) -> float:
    """Bound derived from the arithmetic: 1.5 x the drift of the oracle's fp32-
    accumulation mode from its float64 mode, and never below 5e-2."""
    return max(LOGIT_TOL, 1.5 * float(np.abs(o64 - o32).max()))


def compare_request(o_logits: np.ndarray, g_logits: np.ndarray, drafts, o_accept: int,
                    o_next: int, g_accept: int, g_next: int, report: List[str], tag: str,
                    tol: float = LOGIT_TOL) -> Dict:
    """o_* from the oracle, g_* from the GPU; logits rows 0..n (n = len(drafts))."""
    n = len(drafts)
    d = np.abs(o_logits[: n + 1] - g_logits[: n + 1])
    err = float(d.max())
    assert np.isfinite(g_logits[: n + 1]).all(), f"{tag}: non-finite GPU logits"
    assert err <= tol, f"{tag}: logits max-abs error {err:.4g} > {tol:.4g}"
    gap = top2_gap(o_logits[: n + 1])
    g_greedy = argmax_lowest(g_logits[: n + 1])
    o_greedy = argmax_lowest(o_logits[: n + 1])
    row_err = d.max(axis=1)
    for i in range(n + 1):
        if g_greedy[i] != o_greedy[i]:
            assert gap[i] <= 2 * row_err[i] + 1e-6, \
                f"{tag}: row {i} argmax differs although every logit is within half the gap " \
                f"(gap {gap[i]:.4g}, row err {row_err[i]:.3g})"
            report.append(f"{tag}: row {i} near-tie, oracle gap {gap[i]:.3g}")
    # the GPU's own acceptance must follow from its greedy rows
    from oracle.accept import accept_length
    a = accept_length(drafts, g_greedy)
    assert (g_accept, g_next) == (a, int(g_greedy[a])), f"{tag}: GPU accept/next inconsistent"
    if (g_greedy[: n + 1] == o_greedy[: n + 1]).all():
        assert (g_accept, g_next) == (o_accept, o_next), f"{tag}: accept/next differ from the oracle"
    else:
        report.append(f"{tag}: accept/next ({g_accept},{g_next}) vs oracle ({o_accept},{o_next}) at a near-tie")
    return {"err": err, "min_gap": float(gap.min())}


def shared_units(rows, rb):
    """Runs of consecutive siblings whose live rows fit one row block together
    (the packing the step setup does); returns the run lengths."""
    runs, cur, n = [], 0, 0
    for r in rows:
        if n and cur + r > rb:
            runs.append(n)
            cur, n = 0, 0
        cur += r
        n += 1
    return runs + [n]
