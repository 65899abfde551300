"""Sampled verification -- oracle (test infrastructure only).

The paper's rollouts sample (Evaluation: temperature 1.0, top-p 1.0, top-k
200) and require speculation to be lossless (Introduction; Background, "Why
Workload Matters"); it cites speculative sampling (Leviathan et al. 2023; Chen
et al. 2023) but states no rule of its own.  Reading: the standard lossless
rule for a deterministic drafter (the suffix drafter proposes one token per
position, a point mass q = delta_d):

  target distribution of a row: keep the top_k largest logits (order: value
      descending, then token id ascending), p = softmax(z_kept / T), 0 elsewhere;
  the draft d at row i is accepted with probability min(1, p_i(d) / q(d)) =
      p_i(d), i.e. iff u_i < p_i(d) for a uniform u_i in [0, 1);
  at the first rejection the next token is drawn from the residual
      max(0, p_i - q), normalised = p_i with d removed;
  when every draft is accepted, the next token is drawn from p_n (the bonus
      position).

A draw from weights w with a uniform v in [0, 1) is the inverse CDF in token-id
order: the smallest token t with sum_{s <= t} w_s > v * sum_s w_s.  The
uniforms are inputs (two per row: the acceptance test, then the draw).

Everything is float64.
"""
from __future__ import annotations

from typing import Dict, Sequence

import numpy as np


def kept_tokens(z: np.ndarray, top_k: int) -> np.ndarray:
    """Token ids of the top_k largest logits (value descending, then id ascending)."""
    z = np.asarray(z, dtype=np.float64)
    order = np.lexsort((np.arange(z.size), -z))      # primary: -z, secondary: id
    return np.sort(order[: min(top_k, z.size)])


def filtered_probs(z: np.ndarray, temperature: float, top_k: int) -> np.ndarray:
    """The row's target distribution over the whole vocabulary."""
    z = np.asarray(z, dtype=np.float64)
    keep = kept_tokens(z, top_k)
    s = z[keep] / temperature
    e = np.exp(s - s.max())
    p = np.zeros(z.size)
    p[keep] = e / e.sum()
    return p


def inverse_cdf(w: np.ndarray, v: float) -> int:
    """Smallest token t with sum_{s <= t} w_s > v * sum(w)."""
    c = np.cumsum(np.asarray(w, dtype=np.float64))
    return int(np.searchsorted(c, v * c[-1], side="right"))


def verify_sampled(logits: np.ndarray, drafts: Sequence[int], u_accept: Sequence[float],
                   u_draw: Sequence[float], temperature: float, top_k: int) -> Dict:
    """logits [n+1, V] of the rows [x, d_1..d_n]; returns accept a (drafts kept),
    next token, and per-decision margins (how far each uniform is from the
    boundary that decides it, in probability units)."""
    n = len(drafts)
    margins = []
    for i in range(n + 1):
        p = filtered_probs(logits[i], temperature, top_k)
        if i < n:
            d = int(drafts[i])
            margins.append(abs(u_accept[i] - p[d]))
            if u_accept[i] < p[d]:
                continue
            w = p.copy()
            w[d] = 0.0
        else:
            w = p
        t = inverse_cdf(w, u_draw[i])
        c = np.cumsum(w) / w.sum()
        lo = c[t - 1] if t > 0 else 0.0
        margins.append(min(u_draw[i] - lo, c[t] - u_draw[i]))
        return {"accept": i, "next": t, "margins": margins}
    raise AssertionError("unreachable")
