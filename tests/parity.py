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
(a near-tie), which is reported instead of failed.  A flip at a row whose
oracle gap is 0.1 or more always fails, and so does one whose gap exceeds
twice the row's measured max |logit error| (with every logit within half the
gap the argmax cannot change).  At full depth the logit error can exceed
0.05, so rows whose gap lies in [0.1, 2 x row error) could flip without
breaking the arithmetic: they are counted ("band") and reported, and a flip
there still fails.
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np

from oracle.accept import argmax_lowest, top2_gap
from oracle.sampling import filtered_probs

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
    flips = 0
    band = int(((gap >= NEAR_TIE) & (gap < 2 * row_err)).sum())
    if band:
        report.append(f"{tag}: {band} row(s) with oracle gap in [0.1, 2 x row error)")
    for i in range(n + 1):
        if g_greedy[i] != o_greedy[i]:
            assert gap[i] < NEAR_TIE, \
                f"{tag}: row {i} argmax differs at oracle gap {gap[i]:.4g} >= {NEAR_TIE}"
            assert gap[i] <= 2 * row_err[i] + 1e-6, \
                f"{tag}: row {i} argmax differs although every logit is within half the gap " \
                f"(gap {gap[i]:.4g}, row err {row_err[i]:.3g})"
            flips += 1
            report.append(f"{tag}: row {i} near-tie, oracle gap {gap[i]:.3g}")
    # the GPU's own acceptance must follow from its greedy rows
    from oracle.accept import accept_length
    a = accept_length(drafts, g_greedy)
    assert (g_accept, g_next) == (a, int(g_greedy[a])), f"{tag}: GPU accept/next inconsistent"
    same = (g_accept, g_next) == (o_accept, o_next)
    if (g_greedy[: n + 1] == o_greedy[: n + 1]).all():
        assert same, f"{tag}: accept/next differ from the oracle"
    elif not same:
        report.append(f"{tag}: accept/next ({g_accept},{g_next}) vs oracle ({o_accept},{o_next}) at a near-tie")
    return {"err": err, "min_gap": float(gap.min()), "band": band, "flips": flips, "same": same}


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


def tree_path_brute(tokens, parents, greedy):
    """Accepted path of a draft tree by enumerating every root-to-node path:
    the longest whose every node carries its parent's greedy token, the lowest
    end node among equally long ones.  tokens[0] is the root's token."""
    best = []
    for j in range(len(tokens)):
        path, c = [], j
        while c != 0:
            path.append(c)
            c = parents[c - 1]
        path = path[::-1]
        prev = [0] + path
        if all(tokens[c] == greedy[prev[k]] for k, c in enumerate(path)) and len(path) > len(best):
            best = path
    return best


def compare_tree_request(o: Dict, g_logits: np.ndarray, tokens, parents, g_accept: int, g_next: int,
                         g_path, report: List[str], tag: str, tol: float = LOGIT_TOL) -> bool:
    """o = the oracle's tree verification; g_* from the GPU.  Returns whether
    the GPU took the oracle's path."""
    n = len(tokens) - 1
    d = np.abs(o["logits"] - g_logits[: n + 1])
    err = float(d.max())
    assert np.isfinite(g_logits[: n + 1]).all(), f"{tag}: non-finite GPU logits"
    assert err <= tol, f"{tag}: logits max-abs error {err:.4g} > {tol:.4g}"
    gap = top2_gap(o["logits"])
    g_greedy = argmax_lowest(g_logits[: n + 1])
    o_greedy = argmax_lowest(o["logits"])
    row_err = d.max(axis=1)
    for i in range(n + 1):
        if g_greedy[i] != o_greedy[i]:
            assert gap[i] < NEAR_TIE, f"{tag}: node {i} argmax differs at oracle gap {gap[i]:.4g} >= {NEAR_TIE}"
            assert gap[i] <= 2 * row_err[i] + 1e-6, \
                f"{tag}: node {i} argmax differs although every logit is within half the gap"
            report.append(f"{tag}: node {i} near-tie, oracle gap {gap[i]:.3g}")
    # the GPU's acceptance must follow from its own greedy rows
    want = tree_path_brute(tokens, parents, g_greedy)
    assert list(g_path) == want, f"{tag}: GPU path {list(g_path)} != {want} from its own argmax"
    assert (g_accept, g_next) == (len(want), int(g_greedy[([0] + want)[-1]])), f"{tag}: accept/next"
    if (g_greedy == o_greedy).all():
        assert list(g_path) == o["path"] and g_next == o["next"], f"{tag}: path differs from the oracle"
        return True
    report.append(f"{tag}: path {list(g_path)} vs oracle {o['path']} at a near-tie")
    return list(g_path) == o["path"]


def near_sampled_decision(logits, T, top_k, err, margins) -> bool:
    """True if a logit error of `err` could change one of the sampled decisions
    on the oracle's path: some margin (in probability) is below the bound
    exp(2 err / T) - 1 on how far the error moves a probability or a cumulative
    sum, plus twice the probability mass of the kept tokens within 2 err of the
    top_k boundary (the kept set itself may change there)."""
    delta = np.expm1(2 * err / T) + 1e-5
    for i in range(len(margins)):
        z = logits[min(i, len(logits) - 1)]
        zs = np.sort(z)[::-1]
        if top_k < z.size:
            kth = zs[top_k - 1]
            p = filtered_probs(z, T, top_k)
            delta_i = delta + 2 * p[np.abs(z - kth) < 2 * err].sum()
        else:
            delta_i = delta
        if margins[i] < delta_i:
            return True
    return False
