"""Exact argmax ties on the GPU: ties go to the lowest token id (greedy
verification takes the target's argmax; among equal logits the lowest id).

Two rows of the LM head that hold the same weights give bit-identical logits
on both sides (the same dot product, computed the same way), so ties are
planted by copying rows of W_lm.  For each request, the argmax g of its first
row (whose hidden state does not depend on W_lm) is moved: rows t_lo < t_hi
receive g's weights and row g receives the weights of that row's smallest
logit.  The row's maximum is then attained exactly at t_lo and t_hi, and the
oracle's logits are the original ones with the moved columns copied (exact by
construction).  The pair's placement decides which comparison of the argmax
reduction the tie meets:
  * tiny vocabulary (4096, 32 column blocks of 128): the same 16-column
    matrix-core tile, the two tiles of one wave, two waves of one block, two
    blocks;
  * full vocabulary (151936, 1187 blocks, reduced to 2 layers): blocks that
    the acceptance kernel's threads meet in different waves with the lower id
    in the later wave, in one thread's sequential loop, and in different
    threads of different waves.
The drafts are the oracle's greedy continuation under the planted head, so a
tie resolved to the higher id rejects the first draft; tree drafts carry t_hi
and t_lo as sibling children of the root.
"""
import numpy as np
import pytest
import torch

from oracle.accept import argmax_lowest
from oracle.decoder import RequestKV, Weights, forward_block
from paper_2607_17299_amd import harness, synth
from parity import compare_request

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _war():
    from paper_2607_17299_amd import war
    return war


def _t(a):
    return torch.as_tensor(np.asarray(a), dtype=torch.int32).to(DEV)


class Planted:
    """Logits under the moved LM-head rows: column t takes column moves[t]."""

    def __init__(self, w_lm64: np.ndarray, moves):
        self.w, self.moves = w_lm64, dict(moves)

    def logits(self, hf: np.ndarray) -> np.ndarray:
        z0 = hf @ self.w.T
        z = z0.copy()
        for t, src in self.moves.items():
            z[..., t] = z0[..., src]
        return z

    def weights(self, w_lm: torch.Tensor) -> torch.Tensor:
        out = w_lm.clone()
        for t, src in self.moves.items():
            out[t] = w_lm[src]
        return out


def _hf(cfg, W, kv, tokens):
    hf, _ = forward_block(cfg, W, tokens, kv.length, kv.get, want_logits=False)
    return hf


def _plan(cfg, W, kvs, lasts, pairs):
    """Moves for every request: its row-0 argmax g -> (t_lo, t_hi), g -> its
    row's smallest logit.  Returns the moves and each request's g."""
    w_lm = W.get("w_lm")
    moves, gs, used = {}, [], set()
    for b, (kv, x) in enumerate(zip(kvs, lasts)):
        z = _hf(cfg, W, kv, [x])[0] @ w_lm.T
        g, gmin = int(np.argmax(z)), int(np.argmin(z))
        t_lo, t_hi = pairs[b]
        assert len({g, gmin, t_lo, t_hi} | used) == len(used) + 4, "planted columns collide"
        used |= {g, gmin, t_lo, t_hi}
        moves.update({t_lo: g, t_hi: g, g: gmin})
        gs.append(g)
    return moves, gs


def _greedy_chain(cfg, W, pl: Planted, kv, x, k):
    """k drafts = the greedy continuation under the planted head, then next."""
    toks = [x]
    for _ in range(k + 1):
        z = pl.logits(_hf(cfg, W, kv, toks)[-1:])
        toks.append(int(argmax_lowest(z)[0]))
    return toks[1:k + 1], toks[k + 1]


def _run(cfg, war, model, pool, W, pl, kvs, lasts, ctxs, pairs, k):
    """Chain verify (commit discarded), then a tree verify, both against the
    planted oracle; returns nothing, asserts everything."""
    B = len(kvs)
    seq = _t(range(B))
    ctx = _t(ctxs)
    chains = [_greedy_chain(cfg, W, pl, kvs[b], lasts[b], k) for b in range(B)]
    for b in range(B):
        assert chains[b][0][0] == pairs[b][0]          # the oracle's tie went to t_lo
    dt = _t([c[0] for c in chains])
    acc, nxt = _t([0] * B), _t([0] * B)
    logits = torch.full((B * (k + 1), cfg.vocab), float("nan"), device=DEV)
    war.verify_step(model, pool, seq, ctx, _t(lasts), dt, None, k, acc, nxt, logits)
    war.kv_commit(pool, seq, ctx, _t([-1] * B))
    torch.cuda.synchronize()
    glog = logits.cpu().numpy().reshape(B, k + 1, cfg.vocab)
    report = []
    g_acc = acc.cpu().tolist()
    same = []
    for b in range(B):
        t_lo, t_hi = pairs[b]
        assert glog[b, 0, t_lo] == glog[b, 0, t_hi], "the planted tie is not exact on the GPU"
        assert glog[b, 0, t_lo] == glog[b, 0].max()
        o = pl.logits(_hf(cfg, W, kvs[b], [lasts[b]] + chains[b][0]))
        s = compare_request(o, glog[b], chains[b][0], k, chains[b][1], g_acc[b], int(nxt[b]), report,
                            f"req {b}")
        # the planted tie went to t_lo: the first draft is accepted (a later row
        # may still differ at a reported near-tie of its own)
        assert g_acc[b] >= 1, (b, report)
        if s["same"]:
            assert g_acc[b] == k
        same.append(s["same"])
    print(f"\nplanted ties, chain: accept {g_acc}; reported {report}")
    # tree: root children t_hi (node 1) and t_lo (node 2); node 3 continues t_lo
    # with the greedy chain, node 4 continues t_hi with the same token
    toks = [[p[1], p[0], c[0][1], c[0][1]] for p, c in zip(pairs, chains)]
    parents = [[0, 0, 2, 1]] * B
    acc, nxt, path = _t([0] * B), _t([0] * B), _t(np.zeros((B, 4)))
    war.verify_step_tree(model, pool, seq, ctx, _t(lasts), _t(toks), _t(parents), None, 4, acc, nxt, path)
    war.kv_commit(pool, seq, ctx, _t([-1] * B))
    torch.cuda.synchronize()
    want_next = [int(argmax_lowest(pl.logits(_hf(cfg, W, kvs[b], [lasts[b]] + chains[b][0][:2])))[-1])
                 for b in range(B)]
    t_acc, t_next, t_path = acc.cpu().tolist(), nxt.cpu().tolist(), path.cpu().tolist()
    for b in range(B):
        assert t_path[b][0] == 2, (b, t_path[b])        # the root's tie went to t_lo (node 2)
        if g_acc[b] >= 2:                                # no near-tie at the chain's row 1
            assert t_acc[b] == 2 and t_path[b] == [2, 3, -1, -1], b
        if same[b]:                                      # node 3's row is the chain's row 2
            assert t_next[b] == want_next[b], b


def test_tiny_ties_inside_a_column_block():
    war = _war()
    cfg = synth.TINY
    w_cpu = synth.model_weights(cfg, seed=3, norm_std=0.1)
    W = Weights(cfg, w_cpu)
    ctxs = [150, 171, 96, 230]
    B = len(ctxs)
    seqs = [synth.uniform_tokens(600 + b, n, cfg.vocab) for b, n in enumerate(ctxs)]
    lasts = [int(x) for x in synth.uniform_tokens(650, B, cfg.vocab)]
    kvs = []
    for c in seqs:
        kv = RequestKV(cfg)
        _, new_kv = forward_block(cfg, W, [int(t) for t in c], 0, kv.get, want_logits=False)
        kv.append(new_kv, len(c))
        kvs.append(kv)
    # block 9 = columns 1152..1279; wave w = columns +32w; tile = +16
    pairs = [(9 * 128 + 3, 9 * 128 + 9),            # one 16-column tile
             (13 * 128 + 5, 13 * 128 + 16 + 2),     # the two tiles of one wave
             (17 * 128 + 7, 17 * 128 + 96 + 1),     # waves 0 and 3 of one block
             (21 * 128 + 11, 30 * 128 + 11)]        # two blocks
    moves, _ = _plan(cfg, W, kvs, lasts, pairs)
    pl = Planted(W.get("w_lm"), moves)
    w_gpu = {k: v.to(DEV) for k, v in w_cpu.items()}
    w_gpu["w_lm"] = pl.weights(w_gpu["w_lm"])
    model = war.Model(cfg, w_gpu, max_rows=64)
    pool = war.Pool(cfg, 128, B, 32)
    ctx = _t([0] * B)
    war.prefill_append(model, pool, _t(range(B)), ctx, ctxs, _t(np.concatenate(seqs)), _t([0] * B))
    torch.cuda.synchronize()
    _run(cfg, war, model, pool, W, pl, kvs, lasts, ctxs, pairs, 3)


def test_full_vocabulary_ties_across_the_acceptance_reduction():
    """2 layers at full widths, vocabulary 151936: the acceptance kernel's
    thread c scans column blocks c, c + 256, ... and merges 4 waves."""
    war = _war()
    cfg = synth.reduced(synth.LARGE, 2)
    w = harness.large_weights(cfg)
    W = Weights(cfg, w)
    ctxs = [300, 517, 64]
    B = len(ctxs)
    kv_seed = 9

    def kv_of(b):
        layers = []
        for l in range(cfg.n_layers):
            a = synth.kv_context(cfg, kv_seed, b, l, 0, ctxs[b], DEV).cpu().double().numpy()
            layers.append((a[0], a[1]))
        return RequestKV(cfg, layers)
    kvs = [kv_of(b) for b in range(B)]
    lasts = [int(x) for x in synth.uniform_tokens(660, B, cfg.vocab)]
    pairs = [(255 * 128 + 4, 256 * 128 + 4),        # lower id in thread 255 (wave 3), higher in thread 0
             (10 * 128 + 70, 266 * 128 + 70),       # one thread's sequential scan
             (300 * 128 + 1, 1100 * 128 + 127)]     # thread 44 (wave 0) and thread 76 (wave 1)
    moves, _ = _plan(cfg, W, kvs, lasts, pairs)
    pl = Planted(W.get("w_lm"), moves)
    w2 = dict(w)
    w2["w_lm"] = pl.weights(w["w_lm"])
    model = war.Model(cfg, w2, max_rows=64)
    del w2
    pool = harness.make_pool(cfg, np.array(ctxs), 6)
    harness.load_contexts(pool, cfg, np.array(ctxs), np.arange(B), kv_seed)
    _run(cfg, war, model, pool, W, pl, kvs, lasts, ctxs, pairs, 2)
