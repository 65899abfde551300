"""Synthetic rollout workloads for the verify step (test and benchmark harness).

Builds, on one GPU, the state a verify step starts from: the decoder weights, a
KV pool with each request's cached context, and the step's inputs (pending
tokens and draft tokens from the host suffix drafter).  Everything is seeded.
The cached context's keys and values are imported through ``war_kv_load`` from
the seeded generator rather than recomputed by a prefill: the verify step's
cost and arithmetic do not depend on how the cache was produced, and a prefill
over hundreds of thousands of tokens would dominate every run.

Workloads (the paper's setting; its SWE dataset and Qwen3-32B are not available):
  low_load     8 requests x 32768 cached tokens built from recurring tool-call-
               like motifs, k = 8 drafts from the suffix drafter over 64 prior
               trajectories (System Design, "SuffixDecoding"; Evaluation).
  high_load    64 requests, long-tailed lognormal contexts (median 8192,
               sigma 0.8, clipped to [1024, 65536]), k = 0: plain batched decode.
  high_load_k2 the same contexts, k = 2 drafts taken from a sibling rollout's
               continuation with ~30% of the positions corrupted, so that
               rejected slots are rolled back.
  multi_turn   16 trajectories in 4 groups sharing an 8192-token prefix,
               24576 cached tokens each; a 2048-token observation is appended
               with war_prefill_append, then one k = 4 verify step.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np
import torch

from . import synth, war
from .drafter import SuffixDrafter

LARGE_SEED = 1


def cdiv(a: int, b: int) -> int:
    return -(-a // b)


def large_weights(cfg: synth.ModelConfig = synth.LARGE, device="cuda", seed: int = LARGE_SEED,
                  lm_std: float = synth.WEIGHT_STD) -> Dict[str, torch.Tensor]:
    return synth.model_weights(cfg, seed, device=device, lm_std=lm_std)


@dataclasses.dataclass
class Step:
    """Inputs of one verify step, as host arrays."""
    seq_ids: np.ndarray
    ctx_lens: np.ndarray
    last_tokens: np.ndarray
    drafts: List[List[int]]
    k_max: int
    parents: Optional[List[List[int]]] = None   # tree drafts: parent of node i+1 in [0, i]

    @property
    def B(self) -> int:
        return len(self.seq_ids)

    def draft_array(self) -> np.ndarray:
        a = np.zeros((self.B, max(self.k_max, 1)), np.int32)
        for b, d in enumerate(self.drafts):
            a[b, : len(d)] = d
        return a

    def parent_array(self) -> np.ndarray:
        a = np.zeros((self.B, max(self.k_max, 1)), np.int32)
        for b, p in enumerate(self.parents):
            a[b, : len(p)] = p
        return a

    def draft_lens(self) -> np.ndarray:
        return np.array([len(d) for d in self.drafts], np.int32)

    def rows(self) -> int:
        return int(sum(len(d) + 1 for d in self.drafts))


class DeviceStep:
    """Device copies of a Step plus output buffers."""

    def __init__(self, st: Step, device="cuda", with_logits: bool = False, vocab: int = 0):
        t = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.int32).to(device)
        self.step = st
        self.seq = t(st.seq_ids)
        self.ctx = t(st.ctx_lens)
        self.last = t(st.last_tokens)
        self.drafts = t(st.draft_array())
        self.dlens = t(st.draft_lens())
        self.accept = torch.zeros(st.B, dtype=torch.int32, device=device)
        self.next = torch.zeros(st.B, dtype=torch.int32, device=device)
        self.discard = torch.full((st.B,), -1, dtype=torch.int32, device=device)
        self.logits = (torch.empty((st.B * (st.k_max + 1), vocab), dtype=torch.float32, device=device)
                       if with_logits else None)
        self.parents = t(st.parent_array()) if st.parents is not None else None
        self.path = (torch.full((st.B, max(st.k_max, 1)), -1, dtype=torch.int32, device=device)
                     if st.parents is not None else None)

    def verify(self, model: war.Model, pool: war.Pool, logits: bool = False):
        war.verify_step(model, pool, self.seq, self.ctx, self.last, self.drafts, self.dlens,
                        self.step.k_max, self.accept, self.next, self.logits if logits else None)

    def verify_tree(self, model: war.Model, pool: war.Pool, logits: bool = False):
        war.verify_step_tree(model, pool, self.seq, self.ctx, self.last, self.drafts, self.parents, self.dlens,
                             self.step.k_max, self.accept, self.next, self.path,
                             self.logits if logits else None)

    def run(self, model: war.Model, pool: war.Pool, logits: bool = False):
        """The step's verify call: tree drafts when the step has parents."""
        if self.parents is not None:
            self.verify_tree(model, pool, logits)
        else:
            self.verify(model, pool, logits)

    def verify_sampled(self, model: war.Model, pool: war.Pool, uniforms: torch.Tensor,
                       temperature: float = 1.0, top_k: int = 200):
        war.verify_step_sampled(model, pool, self.seq, self.ctx, self.last, self.drafts, self.dlens,
                                self.step.k_max, uniforms, temperature, top_k, self.accept, self.next)

    def commit(self, pool: war.Pool, discard: bool = True):
        war.kv_commit(pool, self.seq, self.ctx, self.discard if discard else self.accept)


def make_pool(cfg: synth.ModelConfig, ctx_lens, k_max: int, extra_pages: int = 64,
              max_seqs: Optional[int] = None) -> war.Pool:
    P = cfg.page_size
    need = sum(cdiv(int(c) + k_max + 1, P) for c in ctx_lens) + extra_pages
    max_pages = cdiv(int(max(ctx_lens)) + max(k_max, 64) + 1, P)
    return war.Pool(cfg, need, max_seqs or len(ctx_lens), max_pages)


def load_contexts(pool: war.Pool, cfg: synth.ModelConfig, ctx_lens, seq_ids, kv_seed: int,
                  kv_keys=None) -> None:
    """Reserve and fill each sequence's cached context with seeded keys/values."""
    pool.alloc([int(s) for s in seq_ids], [int(c) for c in ctx_lens])
    for i, (s, c) in enumerate(zip(seq_ids, ctx_lens)):
        key = int(kv_keys[i]) if kv_keys is not None else int(s)
        for l in range(cfg.n_layers):
            pool.load(int(s), l, 0, synth.kv_context(cfg, kv_seed, key, l, 0, int(c), "cuda"))
    torch.cuda.synchronize()


# ------------------------------------------------------------------ workloads
def low_load_tokens(seed: int = 2, B: int = 8, ctx: int = 32768, n_prior: int = 64,
                    prior_len: int = 32768, vocab: int = 151936):
    """Motif-built contexts (+1 pending token each) and prior trajectories."""
    bank = synth.MotifBank(seed, vocab)
    contexts = [bank.trajectory(seed * 1000 + b, ctx + 1, end_mid_motif=(b % 2 == 0)) for b in range(B)]
    prior = [bank.trajectory(seed * 1000 + 500 + i, prior_len) for i in range(n_prior)]
    return contexts, prior


def low_load_step(seed: int = 2, B: int = 8, ctx: int = 32768, k: int = 8, n_prior: int = 64,
                  vocab: int = 151936, siblings: Optional[List[List[int]]] = None,
                  sibling_sets: Optional[List[List[List[int]]]] = None, tree: bool = False) -> Step:
    """siblings: per request, one sibling rollout's continuation of the same
    context (GRPO siblings); sibling_sets: several per request.  tree: draft
    trees of up to k nodes instead of k-token chains."""
    contexts, prior = low_load_tokens(seed, B, ctx, n_prior, ctx, vocab)
    d = SuffixDrafter()
    for p in prior:
        d.add_trajectory(p)
    sets = sibling_sets or ([[s] for s in siblings] if siblings is not None else None)
    if sets is not None:
        for b in range(B):
            for sib in sets[b]:
                d.add_trajectory(np.concatenate([contexts[b][-64:], sib]))
    last = np.array([c[-1] for c in contexts], np.int32)
    if tree:
        trees = [d.propose_tree(contexts[b], k) for b in range(B)]
        return Step(np.arange(B, dtype=np.int32), np.full(B, ctx, np.int32), last,
                    [t[0] for t in trees], k, [t[1] for t in trees])
    drafts = [d.propose(contexts[b], k) for b in range(B)]
    return Step(np.arange(B, dtype=np.int32), np.full(B, ctx, np.int32), last, drafts, k)


def time_low_load_drafter(seed: int = 2, B: int = 8, ctx: int = 32768, k: int = 8, n_prior: int = 64,
                          vocab: int = 151936, reps: int = 5) -> dict:
    """Host cost of the low-load drafts (the suffix drafter is harness logic,
    outside the verify step): building the index over the prior trajectories
    once, and proposing k drafts for the B requests (median of `reps`)."""
    import time
    contexts, prior = low_load_tokens(seed, B, ctx, n_prior, ctx, vocab)
    d = SuffixDrafter()
    for p in prior:
        d.add_trajectory(p)
    t0 = time.perf_counter()
    d._build()
    build_ms = (time.perf_counter() - t0) * 1e3
    times = []
    for _ in range(reps):
        t0 = time.perf_counter()
        for b in range(B):
            d.propose(contexts[b], k)
        times.append((time.perf_counter() - t0) * 1e3)
    return {"index_build_ms": round(build_ms, 2), "propose_batch_ms": round(float(np.median(times)), 3),
            "corpus_tokens": int(sum(len(p) for p in prior)), "requests": B, "k": k}


def diverging_siblings(cont: List[List[int]], seed: int, vocab: int) -> List[List[List[int]]]:
    """Three sibling continuations per request, added in this order: one that
    leaves the target's continuation at its first token, one that leaves it at
    its third, and the target's own."""
    rng = np.random.default_rng([seed, 43])
    out = []
    for c in cont:
        a, b = list(c), list(c)
        a[0] = (a[0] + 1 + int(rng.integers(vocab - 1))) % vocab
        if len(b) > 2:
            b[2] = (b[2] + 1 + int(rng.integers(vocab - 1))) % vocab
        out.append([a, b, list(c)])
    return out


def high_load_step(seed: int = 0, B: int = 64, k: int = 0, vocab: int = 151936,
                   drafts: Optional[List[List[int]]] = None) -> Step:
    ctx = synth.lognormal_contexts(seed, B).astype(np.int32)
    last = synth.uniform_tokens(seed + 77, B, vocab)
    return Step(np.arange(B, dtype=np.int32), ctx, last, drafts or [[] for _ in range(B)], k)


def teacher_continuation(model: war.Model, pool: war.Pool, st: Step, n: int) -> List[List[int]]:
    """The target's own greedy continuation of each request (n tokens after the
    pending token), by verify steps that feed back the known prefix and
    discard: the state of the pool is unchanged afterwards.  Every step has
    the same shape (n drafts per request, the unknown tail padded), so a row's
    logits do not depend on the step (steps of different shapes sum in other
    orders and may disagree on an argmax at a near-tie).  Should a fed-back
    prefix still not be accepted in full, the request continues from that
    step's own decision."""
    vocab = model.cfg.vocab
    cont: List[List[int]] = [[] for _ in range(st.B)]
    for _ in range(2 * n + 2):
        if all(len(c) >= n for c in cont):
            break
        drafts = [c[:n] + [(int(st.last_tokens[b]) + 1 + i) % vocab for i in range(n - min(len(c), n))]
                  for b, c in enumerate(cont)]
        ds = DeviceStep(Step(st.seq_ids, st.ctx_lens, st.last_tokens, drafts, n))
        ds.verify(model, pool)
        ds.commit(pool, discard=True)
        nxt = ds.next.cpu().numpy()
        acc = ds.accept.cpu().numpy()
        for b in range(st.B):
            j, a = len(cont[b]), int(acc[b])
            if j >= n:
                continue
            # accepted drafts beyond the known prefix (pads that happen to be
            # greedy) are part of the greedy stream too
            cont[b] = drafts[b][:a] + [int(nxt[b])] if a >= j else cont[b][:a] + [int(nxt[b])]
    assert all(len(c) >= n for c in cont), "the greedy continuation did not settle"
    return [c[:n] for c in cont]


def corrupt(drafts: List[List[int]], p: float, seed: int, vocab: int) -> List[List[int]]:
    mask = synth.bernoulli_mask(seed, (len(drafts), max(len(d) for d in drafts)), p)
    rng = np.random.default_rng([seed, 41])
    out = []
    for b, d in enumerate(drafts):
        out.append([int((x + 1 + rng.integers(vocab - 1)) % vocab) if mask[b, i] else int(x)
                    for i, x in enumerate(d)])
    return out


@dataclasses.dataclass
class MultiTurn:
    """Multi-turn append workload: ``groups`` x ``per_group`` trajectories.  The
    trajectories of a group share a ``prefix``-token cached prefix (forked
    pages), each has ``private`` more cached tokens of its own, and receives an
    ``n_new``-token observation (uniform random ids) through war_prefill_append
    (System Design, "Overview of WAR": a new turn appended to a cached
    trajectory; GRPO siblings share their prompt)."""
    groups: int
    per_group: int
    prefix: int
    private: int
    n_new: int
    obs: List[np.ndarray]

    @property
    def n(self) -> int:
        return self.groups * self.per_group

    @property
    def seq_ids(self) -> np.ndarray:
        return np.arange(self.n, dtype=np.int32)

    @property
    def cached(self) -> int:
        return self.prefix + self.private

    def kv_parts(self, s: int):
        """(generator key, first position, length) of trajectory s's cached context."""
        return [(PREFIX_KEY + s // self.per_group, 0, self.prefix), (s, self.prefix, self.private)]


PREFIX_KEY = 100000


def multi_turn_inputs(seed: int = 5, groups: int = 4, per_group: int = 4, prefix: int = 8192,
                      private: int = 16384, n_new: int = 2048, vocab: int = 151936) -> MultiTurn:
    obs = [synth.uniform_tokens(seed * 1000 + s, n_new, vocab) for s in range(groups * per_group)]
    return MultiTurn(groups, per_group, prefix, private, n_new, obs)


def multi_turn_pool(cfg: synth.ModelConfig, mt: MultiTurn, k_max: int, extra_pages: int = 64) -> war.Pool:
    P = cfg.page_size
    assert mt.prefix % P == 0, "shared prefixes are whole pages"
    own = cdiv(mt.cached + mt.n_new + k_max + 1, P) - mt.prefix // P
    need = mt.groups * (mt.prefix // P) + mt.n * own + extra_pages
    return war.Pool(cfg, need, mt.n, cdiv(mt.cached + mt.n_new + max(k_max, 64) + 1, P))


def load_multi_turn(pool: war.Pool, cfg: synth.ModelConfig, mt: MultiTurn, kv_seed: int) -> None:
    """Each group's prefix is loaded once and forked to its siblings; then every
    trajectory gets its private cached tokens."""
    for g in range(mt.groups):
        s0 = g * mt.per_group
        pool.alloc([s0], [mt.prefix])
        for l in range(cfg.n_layers):
            pool.load(s0, l, 0, synth.kv_context(cfg, kv_seed, PREFIX_KEY + g, l, 0, mt.prefix, "cuda"))
        for j in range(1, mt.per_group):
            pool.fork(s0, s0 + j, mt.prefix)
    pool.alloc([int(s) for s in mt.seq_ids], [mt.cached] * mt.n)
    for s in range(mt.n):
        for l in range(cfg.n_layers):
            pool.load(s, l, mt.prefix, synth.kv_context(cfg, kv_seed, s, l, mt.prefix, mt.private, "cuda"))
    torch.cuda.synchronize()


def multi_turn_kv(cfg: synth.ModelConfig, mt: MultiTurn, kv_seed: int, s: int, layer: int,
                  device="cuda") -> torch.Tensor:
    """[2, Hkv, cached, D] cached keys/values of trajectory s (what the pool holds)."""
    return torch.cat([synth.kv_context(cfg, kv_seed, key, layer, p0, n, device)
                      for key, p0, n in mt.kv_parts(s)], dim=2)


def multi_turn_append(model: war.Model, pool: war.Pool, mt: MultiTurn, last_logits: bool = False):
    """war_prefill_append of every trajectory's observation; returns (next
    tokens, device ctx_lens, last-row logits or None)."""
    t = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.int32).cuda()
    ctx = t(np.full(mt.n, mt.cached, np.int32))
    nxt = t(np.zeros(mt.n, np.int32))
    logits = torch.zeros((mt.n, model.cfg.vocab), device="cuda") if last_logits else None
    war.prefill_append(model, pool, t(mt.seq_ids), ctx, [mt.n_new] * mt.n, t(np.concatenate(mt.obs)),
                       nxt, logits)
    return nxt, ctx, logits


def multi_turn_step(mt: MultiTurn, next_tokens, k: int = 4,
                    siblings: Optional[List[List[int]]] = None) -> Step:
    """The verify step after the append.  Drafts come from the suffix drafter
    over the other trajectories of the same group (their observations, and, when
    given, a sibling rollout that produced each trajectory's continuation)."""
    nxt = np.asarray(next_tokens, np.int32)
    drafts = []
    for s in range(mt.n):
        d = SuffixDrafter()
        g0 = (s // mt.per_group) * mt.per_group
        for j in range(g0, g0 + mt.per_group):
            if j != s:
                d.add_trajectory(mt.obs[j])
        ctx_tokens = np.concatenate([mt.obs[s], nxt[s:s + 1]])
        if siblings is not None:
            d.add_trajectory(np.concatenate([ctx_tokens[-64:], siblings[s]]))
        drafts.append(d.propose(ctx_tokens, k))
    return Step(mt.seq_ids, np.full(mt.n, mt.cached + mt.n_new, np.int32), nxt, drafts, k)


def step_kv_bytes(cfg: synth.ModelConfig, st: Step, shared_prefix: Optional[MultiTurn] = None) -> int:
    """KV bytes one layer's attention must read: every visible key and value.
    With ``shared_prefix`` (forked siblings) a group's common prefix counts
    once: the unique bytes."""
    per_tok = 2 * cfg.n_kv_heads * cfg.head_dim * 2
    toks = int(sum(int(c) + len(d) + 1 for c, d in zip(st.ctx_lens, st.drafts)))
    if shared_prefix is not None:
        mt = shared_prefix
        toks -= (mt.n - mt.groups) * mt.prefix
    return toks * per_tok


def step_bytes(cfg: synth.ModelConfig, st: Step, logits: bool = False,
               shared_prefix: Optional[MultiTurn] = None) -> int:
    """Algorithmic HBM bytes of one verify step: streamed weights, KV read and
    KV written (every layer), logits if written."""
    kv_tok = cfg.kv_bytes_per_token()
    T = st.rows()
    b = cfg.streamed_weight_bytes() + cfg.n_layers * step_kv_bytes(cfg, st, shared_prefix) + T * kv_tok
    if logits:
        b += 4 * T * cfg.vocab
    return b
