"""One verify step and one prefill-append for a batch -- oracle (test infrastructure only).

Composition, per request b with committed length c_b, pending token x_b (the
previous step's emitted token, whose KV is not cached yet) and drafts
d_1..d_n (0 <= n <= k_max):
  1. rows t = [x_b, d_1, ..., d_n] at positions c_b .. c_b + n;
  2. one decoder forward over the rows against the cached context
     (System Design, "SuffixDecoding": verification in one forward pass);
  3. g_i = argmax of row i (ties -> lowest id); a_b = longest prefix of drafts
     with d_m == g_{m-1}; next_b = g_{a_b};
  4. commit: the KV of rows 0..a_b is kept, c_b += a_b + 1, the rest is rolled
     back.  With n = 0 the step is one token of plain batched decode.
Prefill-append (a new turn appended to a cached trajectory, System Design,
"Overview of WAR"): the rows are the new tokens, all of them are committed, and
next_b is the argmax of the last row.

Requests are processed one at a time, so a request's result never depends on
what else is in the batch.

Tree drafts (SuffixDecoding proposes speculation trees; the paper names their
tree-mask handling as a verification cost: Evaluation): node 0 is x_b, node j
(1..n) carries draft token d_j and a parent in 0..j-1.  Node j is scored by
the decoder on its own root-to-node path (the plain definition: exactly what
token-by-token decode along that path computes).  A node is accepted when its
parent is (the root always is) and its token equals the parent's greedy token;
the accepted path ends at the deepest accepted node (ties: the lowest node
index), a_b is its depth and next_b its greedy token.  Without two siblings
carrying the same token this is the walk from the root that follows the one
matching child.  The committed KV is that of the accepted path.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from .accept import accept_length, argmax_lowest
from .decoder import RequestKV, Weights, forward_block


def verify_request(cfg, W: Weights, kv: RequestKV, last_token: int, drafts: Sequence[int],
                   rounding: bool = True, precision: str = "fp64") -> Dict:
    tokens = [int(last_token)] + [int(d) for d in drafts]
    logits, new_kv = forward_block(cfg, W, tokens, kv.length, kv.get, rounding, precision=precision)
    g = argmax_lowest(logits)
    a = accept_length(drafts, g)
    return {"logits": logits, "greedy": g, "accept": a, "next": int(g[a]), "new_kv": new_kv}


def tree_path(parents: Sequence[int], j: int) -> List[int]:
    """Node indices from the root (0) to node j; parents[i-1] is node i's parent."""
    path = [j]
    while path[-1] != 0:
        path.append(int(parents[path[-1] - 1]))
    return path[::-1]


def verify_tree_request(cfg, W: Weights, kv: RequestKV, last_token: int, drafts: Sequence[int],
                        parents: Sequence[int], rounding: bool = True) -> Dict:
    n = len(drafts)
    assert len(parents) == n and all(0 <= int(parents[i]) <= i for i in range(n))
    tok = [int(last_token)] + [int(d) for d in drafts]
    rows = []
    for j in range(n + 1):
        lg, _ = forward_block(cfg, W, [tok[i] for i in tree_path(parents, j)], kv.length, kv.get, rounding)
        rows.append(lg[-1])
    logits = np.stack(rows)
    g = argmax_lowest(logits)
    # a node is accepted when its parent is and its token is the parent's greedy token
    ok, depth = [True] + [False] * n, [0] * (n + 1)
    for j in range(1, n + 1):
        p = int(parents[j - 1])
        ok[j] = ok[p] and tok[j] == int(g[p])
        depth[j] = depth[p] + 1
    cur = max((j for j in range(n + 1) if ok[j]), key=lambda j: (depth[j], -j))
    path = tree_path(parents, cur)[1:]
    _, new_kv = forward_block(cfg, W, [tok[i] for i in [0] + path], kv.length, kv.get, rounding)
    return {"logits": logits, "greedy": g, "accept": len(path), "path": path, "next": int(g[cur]),
            "new_kv": new_kv}


def verify_batch(cfg, W: Weights, kvs: List[RequestKV], last_tokens, drafts: List[Sequence[int]],
                 rounding: bool = True) -> List[Dict]:
    return [verify_request(cfg, W, kv, x, d, rounding) for kv, x, d in zip(kvs, last_tokens, drafts)]


def commit_request(kv: RequestKV, result: Dict, accept: int | None = None) -> None:
    """Keep rows 0..a of the step's new KV (a = -1 keeps nothing)."""
    a = result["accept"] if accept is None else accept
    kv.append(result["new_kv"], a + 1)


def prefill_request(cfg, W: Weights, kv: RequestKV, tokens: Sequence[int],
                    rounding: bool = True) -> Dict:
    logits, new_kv = forward_block(cfg, W, [int(t) for t in tokens], kv.length, kv.get, rounding)
    kv.append(new_kv, len(tokens))
    g = argmax_lowest(logits)
    return {"logits": logits, "greedy": g, "next": int(g[-1])}


def greedy_decode(cfg, W: Weights, kv: RequestKV, last_token: int, steps: int,
                  rounding: bool = True) -> List[int]:
    """Token-by-token greedy decode (k = 0 steps); returns the emitted tokens."""
    out, x = [], int(last_token)
    for _ in range(steps):
        r = verify_request(cfg, W, kv, x, [], rounding)
        commit_request(kv, r)
        x = r["next"]
        out.append(x)
    return out
