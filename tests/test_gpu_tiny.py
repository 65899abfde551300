"""GPU parity on the tiny decoder (2 layers, d 256, 4/2 heads, vocab 4096):
matrix-core lane layout, input generators CPU == GPU, paged-KV bookkeeping
bit-exact against the oracle pool, and the whole prefill -> verify -> commit
path against the oracle (logits, accept lengths, next tokens, KV contents)."""
import copy

import numpy as np
import pytest
import torch

from oracle.accept import argmax_lowest
from oracle.decoder import RequestKV, Weights
from oracle.pages import PagePool
from oracle.verify import commit_request, greedy_decode, prefill_request, verify_request, verify_tree_request
from paper_2607_17299_amd import synth
from paper_2607_17299_amd.drafter import SuffixDrafter
from parity import NEAR_TIE, compare_request, compare_tree_request, near_sampled_decision, shared_units

pytestmark = pytest.mark.gpu
CFG = synth.TINY
DEV = "cuda"


def _war():
    from paper_2607_17299_amd import war
    return war


def test_mfma_lane_layout():
    war = _war()
    g = torch.Generator().manual_seed(0)
    A = torch.randn(16, 32, generator=g).to(torch.bfloat16)
    B = torch.randn(32, 16, generator=g).to(torch.bfloat16)
    C = war.debug_mfma16(A.to(DEV), B.to(DEV)).cpu()
    ref = A.double() @ B.double()
    assert torch.allclose(C.double(), ref, atol=1e-4, rtol=1e-5), (C.double() - ref).abs().max()


def test_generators_identical_on_cpu_and_gpu():
    for shape_cfg, seed in ((CFG, 0), (synth.reduced(synth.LARGE, 1, vocab=1024), 1)):
        for i, (name, shape) in enumerate(synth.weight_shapes(shape_cfg)[:6]):
            a = synth.make_weight(shape_cfg, seed, i, name, shape, "cpu", norm_std=0.1)
            b = synth.make_weight(shape_cfg, seed, i, name, shape, DEV, norm_std=0.1).cpu()
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), name
    a = synth.kv_context(synth.LARGE, 5, 3, 7, 1000, 300, "cpu")
    b = synth.kv_context(synth.LARGE, 5, 3, 7, 1000, 300, DEV).cpu()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


# --------------------------------------------------------------------------- setup
@pytest.fixture(scope="module")
def tiny():
    war = _war()
    w_cpu = synth.model_weights(CFG, seed=0, norm_std=0.1)
    w_gpu = {k: v.to(DEV) for k, v in w_cpu.items()}
    model = war.Model(CFG, w_gpu, max_rows=256)
    return {"war": war, "w_cpu": w_cpu, "W": Weights(CFG, w_cpu), "model": model, "w_gpu": w_gpu}


def _snap_equal(gpu_state, oracle: PagePool, tag=""):
    o = oracle.snapshot()
    np.testing.assert_array_equal(gpu_state["stack"], o["stack"], err_msg=tag + " stack")
    np.testing.assert_array_equal(gpu_state["refcount"], o["refcount"], err_msg=tag + " refcount")
    np.testing.assert_array_equal(gpu_state["held"], o["held"], err_msg=tag + " held")
    np.testing.assert_array_equal(gpu_state["base"], o["base"], err_msg=tag + " base")
    np.testing.assert_array_equal(gpu_state["table"], o["table"], err_msg=tag + " table")


def test_bookkeeping_bit_exact_against_oracle(tiny):
    war, model = tiny["war"], tiny["model"]
    rng = np.random.default_rng(0)
    NP, S, MP = 96, 6, 24
    pool = war.Pool(CFG, NP, S, MP)
    ora = PagePool(NP, 16, S, MP)
    ctx = np.zeros(S, np.int64)
    st = pool.state()
    assert st["status"] == 0
    _snap_equal(st, ora, "init")
    for step in range(40):
        op = int(rng.integers(0, 5))
        ids = rng.permutation(S)[: int(rng.integers(1, S + 1))].tolist()
        tag = f"step {step} op {op}"
        if op == 0:
            n = [int(x) for x in rng.integers(0, 120, len(ids))]
            try:
                ora.alloc(ids, n)
            except Exception:
                with pytest.raises(war.WarError):
                    pool.alloc(ids, n)
                continue
            pool.alloc(ids, n)
            for s in ids:
                ctx[s] = min(ctx[s], int(ora.held[s]) * 16)
        elif op == 1:
            src, dst = int(rng.integers(S)), int(rng.integers(S))
            n = int(rng.integers(0, ora.held[src] + 1)) * 16
            try:
                ora.fork(src, dst, n)
            except Exception:
                with pytest.raises(war.WarError):
                    pool.fork(src, dst, n)
                continue
            pool.fork(src, dst, n)
            ctx[dst] = n
        elif op == 2:
            ora.free(ids)
            pool.free(ids)
            ctx[ids] = 0
        else:
            # a verify step on the tiny model; commit with chosen accept lengths
            k = int(rng.integers(0, 5))
            dl = [int(x) for x in rng.integers(0, k + 1, len(ids))]
            c = [int(ctx[s]) for s in ids]
            try:
                ora.reserve(ids, c, dl)
            except Exception:
                continue   # out of pages: covered by the capacity test
            B = len(ids)
            t = lambda a: torch.tensor(a, dtype=torch.int32, device=DEV)
            drafts = t(rng.integers(0, CFG.vocab, (B, max(k, 1))).tolist())
            acc, nxt = t([0] * B), t([0] * B)
            war.verify_step(model, pool, t(ids), t(c), t(rng.integers(0, CFG.vocab, B).tolist()),
                            drafts, t(dl), k, acc, nxt)
            st = pool.state()
            assert st["status"] == 0, tag
            _snap_equal(st, ora, tag + " reserve")
            choose = [int(rng.integers(-1, d + 1)) for d in dl]
            ctx_d = t(c)
            war.kv_commit(pool, t(ids), ctx_d, t(choose))
            new = ora.commit(ids, c, choose)
            np.testing.assert_array_equal(ctx_d.cpu().numpy(), new, err_msg=tag)
            for s, v in zip(ids, new):
                ctx[s] = int(v)
        st = pool.state()
        assert st["status"] == 0, tag
        _snap_equal(st, ora, tag)
        ora.check_invariants()


def test_out_of_pages_is_reported_without_state_change(tiny):
    war = tiny["war"]
    pool = war.Pool(CFG, 8, 3, 8)
    pool.alloc([0], [100])
    before = pool.state()
    with pytest.raises(war.WarError) as e:
        pool.alloc([1], [64])
    assert e.value.status == -2
    after = pool.state()
    for k in ("stack", "refcount", "held", "table"):
        np.testing.assert_array_equal(before[k], after[k])


# ------------------------------------------------------------- end-to-end parity
def _tiny_workload(seed=1, B=4, ctx_len=512, k=4):
    prior = [synth.uniform_tokens(100 + seed * 10 + i, 1024, CFG.vocab) for i in range(8)]
    ctxs = [synth.uniform_tokens(200 + seed * 10 + b, ctx_len, CFG.vocab) for b in range(B)]
    return prior, ctxs


def _prefill_both(tiny, ctxs, pool_pages=256):
    war, model, W = tiny["war"], tiny["model"], tiny["W"]
    B = len(ctxs)
    pool = war.Pool(CFG, pool_pages, B, 64)
    seq = torch.arange(B, dtype=torch.int32, device=DEV)
    ctx = torch.zeros(B, dtype=torch.int32, device=DEV)
    toks = torch.from_numpy(np.concatenate(ctxs)).to(torch.int32).to(DEV)
    nxt = torch.zeros(B, dtype=torch.int32, device=DEV)
    last = torch.zeros((B, CFG.vocab), dtype=torch.float32, device=DEV)
    war.prefill_append(model, pool, seq, ctx, [len(c) for c in ctxs], toks, nxt, last)
    torch.cuda.synchronize()
    kvs, onext, ologits = [], [], []
    for c in ctxs:
        kv = RequestKV(CFG)
        r = prefill_request(CFG, W, kv, c)
        kvs.append(kv)
        onext.append(r["next"])
        ologits.append(r["logits"][-1])
    return pool, seq, ctx, kvs, np.array(onext), np.stack(ologits), nxt.cpu().numpy(), last.cpu().numpy()


def test_prefill_matches_oracle(tiny):
    _, ctxs = _tiny_workload(seed=1, B=3, ctx_len=300)
    ctxs[1] = ctxs[1][:37]     # ragged: a partial page and a short sequence
    pool, seq, ctx, kvs, onext, ologits, gnext, glogits = _prefill_both(tiny, ctxs)
    assert ctx.cpu().tolist() == [len(c) for c in ctxs]
    err = np.abs(glogits - ologits).max()
    assert err < 5e-2, err
    for b in range(len(ctxs)):
        if gnext[b] != onext[b]:
            gap = np.sort(ologits[b])[-1] - np.sort(ologits[b])[-2]
            assert gap < NEAR_TIE and gap <= 2 * np.abs(glogits[b] - ologits[b]).max() + 1e-6, (b, gap)
        for l in range(CFG.n_layers):
            g = pool.gather_kv(b, len(ctxs[b]), l).double().cpu().numpy()
            K, V = kvs[b].get(l)
            np.testing.assert_allclose(g[0], K, atol=2e-2, rtol=2e-2)
            np.testing.assert_allclose(g[1], V, atol=2e-2, rtol=2e-2)


def _run_steps(tiny, steps, draft_mode, seed, report):
    """Prefill 4 x 512, then `steps` verify+commit steps with drafts from the
    host suffix drafter ('suffix'), the oracle's own greedy continuation
    ('greedy'), or a mix with corrupted positions ('mixed')."""
    war, model, W = tiny["war"], tiny["model"], tiny["W"]
    prior, ctxs = _tiny_workload(seed=seed)
    B, k = len(ctxs), 4
    pool, seq, ctx, kvs, onext, *_ = _prefill_both(tiny, ctxs)
    drafter = SuffixDrafter()
    for p in prior:
        drafter.add_trajectory(p)
    hist = [list(c) for c in ctxs]
    pending = [int(x) for x in onext]          # inputs always come from the oracle side
    rng = np.random.default_rng(seed)
    stats = []
    for step in range(steps):
        drafts = []
        for b in range(B):
            if draft_mode == "suffix":
                d = drafter.propose(hist[b] + [pending[b]], k)
            else:
                d = greedy_decode(CFG, W, copy.deepcopy(kvs[b]), pending[b], k)
                if draft_mode == "mixed":
                    d = [int(rng.integers(CFG.vocab)) if rng.random() < 0.3 else x for x in d]
                d = d[: int(rng.integers(0, k + 1))] if draft_mode == "mixed" else d
            drafts.append(d)
        dl = [len(d) for d in drafts]
        dt = np.zeros((B, k), np.int32)
        for b, d in enumerate(drafts):
            dt[b, : len(d)] = d
        t = lambda a: torch.tensor(np.asarray(a), dtype=torch.int32, device=DEV)
        acc, nxt = t([0] * B), t([0] * B)
        logits = torch.full((B * (k + 1), CFG.vocab), float("nan"), device=DEV)
        war.verify_step(model, pool, seq, ctx, t(pending), t(dt), t(dl), k, acc, nxt, logits)
        torch.cuda.synchronize()
        g_acc, g_nxt = acc.cpu().numpy(), nxt.cpu().numpy()
        glog = logits.cpu().numpy().reshape(B, k + 1, CFG.vocab)
        war.kv_commit(pool, seq, ctx, acc)                # the GPU's own decision
        torch.cuda.synchronize()
        new_pending = []
        for b in range(B):
            r = verify_request(CFG, W, kvs[b], pending[b], drafts[b])
            # fails unless the GPU's decision equals the oracle's or differs at a
            # reported near-tie (oracle gap < 0.1)
            s = compare_request(r["logits"], glog[b], drafts[b], r["accept"], r["next"],
                                int(g_acc[b]), int(g_nxt[b]), report, f"step {step} req {b}")
            stats.append(s)
            # after a reported near-tie the oracle follows the GPU's decision,
            # so that every later step is still compared
            commit_request(kvs[b], r, int(g_acc[b]))
            hist[b] += [pending[b]] + drafts[b][: int(g_acc[b])]
            new_pending.append(int(g_nxt[b]))
        assert ctx.cpu().tolist() == [kv.length for kv in kvs], f"step {step}"
        for b in range(B):
            for l in range(CFG.n_layers):
                g = pool.gather_kv(b, kvs[b].length, l).double().cpu().numpy()
                K, V = kvs[b].get(l)
                np.testing.assert_allclose(g[0], K, atol=2e-2, rtol=2e-2)
                np.testing.assert_allclose(g[1], V, atol=2e-2, rtol=2e-2)
        pending = new_pending
    assert len(stats) == steps * B
    return stats


def _greedy_with_choices(cfg, W, kv, x, n, chosen):
    """Token-by-token greedy decode, except that position j emits chosen[j]
    where given (a near-tie the GPU decided the other way)."""
    out = []
    while len(out) < n:
        r = verify_request(cfg, W, kv, x, [])
        commit_request(kv, r)
        x = chosen.get(len(out), r["next"])
        out.append(x)
    return out


def test_mode_switching_is_stateless(tiny):
    """Consecutive steps with k_max = 0 (plain decode) and k_max > 0 on the same
    pool and sequences (the speculation on/off switch), drafting the oracle's
    own continuation.  The GPU commits its own accept lengths; every step it
    accepts all drafts, except where a row is a reported near-tie (oracle top-2
    gap below 0.1), where the oracle then follows the GPU's choice.  The tokens
    the GPU emits over the whole schedule must be the oracle's token-by-token
    greedy stream with the GPU's choice at those near-ties (and at no other
    position)."""
    war, model, W = tiny["war"], tiny["model"], tiny["W"]
    _, ctxs = _tiny_workload(seed=7, B=3, ctx_len=200)
    pool, seq, ctx, kvs, onext, ologits, gnext, _ = _prefill_both(tiny, ctxs)
    assert (gnext == onext).all()
    start = [RequestKV(CFG, list(kv.layers)) for kv in kvs]
    pending = [int(x) for x in onext]
    emitted = [[] for _ in ctxs]
    chosen = [{} for _ in ctxs]
    report = []
    t = lambda a: torch.tensor(np.asarray(a), dtype=torch.int32, device=DEV)
    for step, k in enumerate([0, 4, 0, 2, 8, 0, 1]):
        drafts = [greedy_decode(CFG, W, copy.deepcopy(kvs[b]), pending[b], k) for b in range(len(ctxs))]
        dt = np.zeros((len(ctxs), max(k, 1)), np.int32)
        for b, d in enumerate(drafts):
            dt[b, :k] = d
        acc, nxt = t([0] * len(ctxs)), t([0] * len(ctxs))
        logits = torch.zeros((len(ctxs) * (k + 1), CFG.vocab), device=DEV)
        war.verify_step(model, pool, seq, ctx, t(pending), t(dt), t([k] * len(ctxs)), k, acc, nxt, logits)
        war.kv_commit(pool, seq, ctx, acc)                # the GPU's own decision
        torch.cuda.synchronize()
        g_acc, g_nxt = acc.cpu().numpy(), nxt.cpu().numpy()
        glog = logits.cpu().numpy().reshape(len(ctxs), k + 1, CFG.vocab)
        for b in range(len(ctxs)):
            r = verify_request(CFG, W, kvs[b], pending[b], drafts[b])
            assert r["accept"] == k                      # the oracle accepts its own continuation
            s = compare_request(r["logits"], glog[b], drafts[b], r["accept"], r["next"], int(g_acc[b]),
                                int(g_nxt[b]), report, f"step {step} (k={k}) req {b}")
            ga, gn = int(g_acc[b]), int(g_nxt[b])
            if s["same"]:
                assert (ga, gn) == (k, r["next"])
            else:                                        # a reported near-tie: row ga flipped
                assert s["flips"] >= 1 and gn != int(r["greedy"][ga])
                chosen[b][len(emitted[b]) + ga] = gn
            commit_request(kvs[b], r, ga)                 # the oracle follows the GPU
            emitted[b] += drafts[b][:ga] + [gn]          # the GPU's emitted tokens
            pending[b] = gn
        assert ctx.cpu().tolist() == [kv.length for kv in kvs]
    print(f"\nmode switching: reported {report}")
    for b in range(len(ctxs)):
        want = _greedy_with_choices(CFG, W, start[b], int(onext[b]), len(emitted[b]), chosen[b])
        assert emitted[b] == want
        g = pool.gather_kv(b, kvs[b].length, CFG.n_layers - 1).double().cpu().numpy()
        K, V = kvs[b].get(CFG.n_layers - 1)
        np.testing.assert_allclose(g[0], K, atol=2e-2, rtol=2e-2)
        np.testing.assert_allclose(g[1], V, atol=2e-2, rtol=2e-2)


def test_shared_prefix_cascade(tiny):
    """Forked siblings: requests 0-2 share a 1056-token prefix (war_kv_fork of
    whole pages) and each appends 100 private tokens; request 3 is unrelated.
    Two verify steps with ragged drafts (2, 1, 4, 4 tokens: the oracle's own
    continuation, request 2 with a wrong second draft): requests 0 and 1 have
    6 + 4 live rows and attend their shared chunk in one unit, request 2 (10
    rows) in its own.  Logits, accepts and the committed KV are compared with
    the oracle, which runs every request on its own."""
    war, model, W = tiny["war"], tiny["model"], tiny["W"]
    prefix = synth.uniform_tokens(901, 1056, CFG.vocab)
    priv = [synth.uniform_tokens(910 + b, 100, CFG.vocab) for b in range(3)] + \
           [synth.uniform_tokens(920, 500, CFG.vocab)]
    B, k = 4, 4
    dls = [2, 1, 4, 4]
    pool = war.Pool(CFG, 512, B, 128)
    t = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.int32).to(DEV)
    c0 = t([0])
    war.prefill_append(model, pool, t([0]), c0, [len(prefix)], t(prefix), t([0]), None)
    for b in (1, 2):
        pool.fork(0, b, len(prefix))
    ctx = t([len(prefix)] * 3 + [0])
    nxt = t([0] * B)
    war.prefill_append(model, pool, t(range(B)), ctx, [len(x) for x in priv], t(np.concatenate(priv)), nxt, None)
    torch.cuda.synchronize()
    bt = pool.block_tables.cpu().numpy()
    assert (bt[1, :66] == bt[0, :66]).all() and (bt[2, :66] == bt[0, :66]).all()
    # oracle: each request on its own
    base = RequestKV(CFG)
    prefill_request(CFG, W, base, prefix)
    kvs, pending = [], []
    for b in range(B):
        kv = RequestKV(CFG, list(base.layers)) if b < 3 else RequestKV(CFG)
        r = prefill_request(CFG, W, kv, priv[b])
        kvs.append(kv)
        pending.append(r["next"])
    seq = t(range(B))
    report = []
    G = CFG.n_q_heads // CFG.n_kv_heads
    assert shared_units([G * (d + 1) for d in dls[:3]], 16) == [2, 1]
    for step in range(2):
        drafts = [greedy_decode(CFG, W, copy.deepcopy(kvs[b]), pending[b], dls[b]) for b in range(B)]
        drafts[2][1] = (drafts[2][1] + 1) % CFG.vocab
        dt = np.zeros((B, k), np.int32)
        for b, d in enumerate(drafts):
            dt[b, :len(d)] = d
        acc, nx = t([0] * B), t([0] * B)
        logits = torch.zeros((B * (k + 1), CFG.vocab), device=DEV)
        war.verify_step(model, pool, seq, ctx, t(pending), t(dt), t(dls), k, acc, nx, logits)
        torch.cuda.synchronize()
        # the plan: 2 chunks of 1024 keys for each sibling, 1 for request 3 (7
        # slots); chunk 0 of requests 0 and 1 is one unit: 6 units
        n_items = war.debug_workspace(model, "n_items", torch.int32, (2,)).cpu().tolist()
        assert n_items == [7, 6], n_items
        g_acc, g_nxt = acc.cpu().numpy(), nx.cpu().numpy()
        glog = logits.cpu().numpy().reshape(B, k + 1, CFG.vocab)
        o_acc = []
        for b in range(B):
            r = verify_request(CFG, W, kvs[b], pending[b], drafts[b])
            compare_request(r["logits"], glog[b], drafts[b], r["accept"], r["next"], int(g_acc[b]),
                            int(g_nxt[b]), report, f"step {step} req {b}")
            commit_request(kvs[b], r)
            pending[b] = r["next"]
            o_acc.append(r["accept"])
        assert o_acc == [2, 1, 1, 4], o_acc
        war.kv_commit(pool, seq, ctx, t(o_acc))
        torch.cuda.synchronize()
        assert ctx.cpu().tolist() == [kv.length for kv in kvs]
    for b in range(B):
        g = pool.gather_kv(b, kvs[b].length, CFG.n_layers - 1).double().cpu().numpy()
        K, V = kvs[b].get(CFG.n_layers - 1)
        np.testing.assert_allclose(g[0], K, atol=2e-2, rtol=2e-2)
        np.testing.assert_allclose(g[1], V, atol=2e-2, rtol=2e-2)
    print(f"\nshared-prefix cascade: reported {report}")


def _tree_drafts(kind, rng, W, kv, pending, hist, drafter, k):
    """(tokens, parents) of one request's draft tree, at most k nodes."""
    if kind == 0:                                   # the host suffix drafter's tree
        return drafter.propose_tree(hist + [pending], k)
    if kind == 1:                                   # the greedy branch among distractors
        g = greedy_decode(CFG, W, copy.deepcopy(kv), pending, 4)
        x = [int(t) for t in rng.integers(0, CFG.vocab, 3)]
        return [x[0], g[0], g[1], x[1], g[2], x[2], g[3]][:k], [0, 0, 2, 2, 3, 1, 5][:k]
    if kind == 2:                                   # a random tree
        n = int(rng.integers(1, k + 1))
        return ([int(t) for t in rng.integers(0, CFG.vocab, n)],
                [int(rng.integers(0, i + 1)) for i in range(n)])
    return [], []                                   # no drafts: one decode row


def test_tree_verification_matches_oracle(tiny):
    """Draft trees (war_verify_step_tree), 4 requests x 512 cached tokens, at
    most 8 nodes: a suffix-drafter tree, the greedy continuation placed among
    distractor branches, a random tree, and no drafts, rotated over 3 steps.
    Node logits, accepted path and next token against the oracle's tree
    verification; after the commit the cache holds exactly the accepted path's
    KV (the step moved it to consecutive slots).  Near-ties are reported; a
    request whose path then differs ends the comparison of later steps."""
    war, model, W = tiny["war"], tiny["model"], tiny["W"]
    prior, ctxs = _tiny_workload(seed=11)
    B, k = len(ctxs), 8
    pool, seq, ctx, kvs, onext, *_ = _prefill_both(tiny, ctxs)
    drafter = SuffixDrafter()
    for p in prior:
        drafter.add_trajectory(p)
    hist = [list(c) for c in ctxs]
    pending = [int(x) for x in onext]
    rng = np.random.default_rng(11)
    t = lambda a: torch.tensor(np.asarray(a), dtype=torch.int32, device=DEV)
    report, greedy_hits = [], 0
    for step in range(3):
        trees = [_tree_drafts((step + b) % 4, rng, W, kvs[b], pending[b], hist[b], drafter, k)
                 for b in range(B)]
        dt, dp = np.zeros((B, k), np.int32), np.zeros((B, k), np.int32)
        for b, (tk, par) in enumerate(trees):
            dt[b, : len(tk)], dp[b, : len(par)] = tk, par
        acc, nxt, path = t([0] * B), t([0] * B), t(np.zeros((B, k)))
        logits = torch.full((B * (k + 1), CFG.vocab), float("nan"), device=DEV)
        ctx_before = ctx.cpu().numpy().copy()
        war.verify_step_tree(model, pool, seq, ctx, t(pending), t(dt), t(dp), t([len(x[0]) for x in trees]),
                             k, acc, nxt, path, logits)
        war.kv_commit(pool, seq, ctx, acc)
        torch.cuda.synchronize()
        g_acc, g_nxt, g_path = acc.cpu().numpy(), nxt.cpu().numpy(), path.cpu().numpy()
        glog = logits.cpu().numpy().reshape(B, k + 1, CFG.vocab)
        same = True
        for b, (tk, par) in enumerate(trees):
            tag = f"step {step} req {b}"
            r = verify_tree_request(CFG, W, kvs[b], pending[b], tk, par)
            a = int(g_acc[b])
            assert (g_path[b, a:] == -1).all(), tag
            ok = compare_tree_request(r, glog[b], [pending[b]] + tk, par, a, int(g_nxt[b]), g_path[b, :a],
                                      report, tag)
            if (step + b) % 4 == 1 and ok:
                assert r["accept"] == 4 and a == 4, tag
                greedy_hits += 1
            if not ok:
                same = False
                continue
            commit_request(kvs[b], r)
            assert int(ctx.cpu()[b]) == kvs[b].length == int(ctx_before[b]) + a + 1, tag
            for l in range(CFG.n_layers):
                g = pool.gather_kv(b, kvs[b].length, l).double().cpu().numpy()
                K, V = kvs[b].get(l)
                np.testing.assert_allclose(g[0], K, atol=2e-2, rtol=2e-2, err_msg=tag)
                np.testing.assert_allclose(g[1], V, atol=2e-2, rtol=2e-2, err_msg=tag)
            hist[b] += [pending[b]] + [tk[i - 1] for i in r["path"]]
            pending[b] = r["next"]
        if not same:
            break
    assert pool.state()["status"] == 0
    assert greedy_hits >= 2
    print(f"\ntree verification: reported {report}")


def test_tree_parent_out_of_range_is_flagged(tiny):
    """A parent outside [0, i) sets the device error flag and is read as i - 1
    (the step then verifies a chain)."""
    war, model, W = tiny["war"], tiny["model"], tiny["W"]
    _, ctxs = _tiny_workload(seed=12, B=1, ctx_len=40)
    pool, seq, ctx, kvs, onext, *_ = _prefill_both(tiny, ctxs, pool_pages=16)
    t = lambda a: torch.tensor(np.asarray(a), dtype=torch.int32, device=DEV)
    g = greedy_decode(CFG, W, copy.deepcopy(kvs[0]), int(onext[0]), 3)
    acc, nxt, path = t([0]), t([0]), t([[0, 0, 0]])
    war.verify_step_tree(model, pool, seq, ctx, t([int(onext[0])]), t([g]), t([[0, 7, 2]]), None, 3,
                         acc, nxt, path)
    torch.cuda.synchronize()
    assert pool.state()["status"] == -5          # WAR_ERR_DEVICE
    a = int(acc.cpu()[0])
    assert path.cpu().tolist()[0] == [1, 2, 3][:a] + [-1] * (3 - a)


@pytest.mark.parametrize("T,top_k", [(1.0, 200), (0.7, 50)])
def test_sampled_verification_matches_oracle(tiny, T, top_k):
    """Three sampled verify steps (k = 4, ragged drafts: the oracle's greedy
    continuation, partly corrupted) against the oracle's sampled rule on the
    oracle's logits with the same uniforms.  With a nearly flat top-k target
    the draw boundaries sit ~1e-3 apart, closer than the logit error can move
    them, so many draws are legitimately near: a decision may differ only where
    the logit error could move it (reported); both sides then continue from
    the oracle's outcome.  The decision kernels themselves are checked exactly
    in test_gpu_sampling.py."""
    war, model, W = tiny["war"], tiny["model"], tiny["W"]
    from oracle.sampling import verify_sampled
    _, ctxs = _tiny_workload(seed=5, B=4, ctx_len=300)
    B, k = len(ctxs), 4
    pool, seq, ctx, kvs, onext, *_ = _prefill_both(tiny, ctxs)
    rng = np.random.default_rng(21)
    pending = [int(x) for x in onext]
    report, checked = [], 0
    t = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.int32).to(DEV)
    for step in range(3):
        drafts = []
        for b in range(B):
            d = greedy_decode(CFG, W, copy.deepcopy(kvs[b]), pending[b], k)
            d = [int(rng.integers(CFG.vocab)) if rng.random() < 0.25 else x for x in d]
            drafts.append(d[: int(rng.integers(0, k + 1))])
        dt = np.zeros((B, k), np.int32)
        for b, d in enumerate(drafts):
            dt[b, :len(d)] = d
        u = rng.random((B * (k + 1), 2)).astype(np.float32)
        acc, nx = t([0] * B), t([0] * B)
        logits = torch.zeros((B * (k + 1), CFG.vocab), device=DEV)
        war.verify_step_sampled(model, pool, seq, ctx, t(pending), t(dt), t([len(d) for d in drafts]), k,
                                torch.from_numpy(u).to(DEV), T, top_k, acc, nx, logits)
        torch.cuda.synchronize()
        g_acc, g_nxt = acc.cpu().numpy(), nx.cpu().numpy()
        glog = logits.cpu().numpy().reshape(B, k + 1, CFG.vocab)
        o_acc = []
        for b in range(B):
            n = len(drafts[b])
            r = verify_request(CFG, W, kvs[b], pending[b], drafts[b])
            uu = u[b * (k + 1): b * (k + 1) + n + 1].astype(np.float64)
            rs = verify_sampled(r["logits"], drafts[b], uu[:, 0], uu[:, 1], T, top_k)
            err = float(np.abs(glog[b, : n + 1] - r["logits"]).max())
            assert err < 5e-2, err
            if (int(g_acc[b]), int(g_nxt[b])) != (rs["accept"], rs["next"]):
                assert near_sampled_decision(r["logits"], T, top_k, err, rs["margins"]), \
                    (step, b, (int(g_acc[b]), int(g_nxt[b])), (rs["accept"], rs["next"]), rs["margins"], err)
                report.append(f"step {step} req {b}: near-boundary sample differs")
            else:
                checked += 1
            commit_request(kvs[b], r, rs["accept"])
            pending[b] = rs["next"]
            o_acc.append(rs["accept"])
        war.kv_commit(pool, seq, ctx, t(o_acc))
        torch.cuda.synchronize()
        assert ctx.cpu().tolist() == [kv.length for kv in kvs]
    print(f"\nsampled T={T} top_k={top_k}: {checked} exact, reported {report}")


def test_sampled_top1_equals_greedy(tiny):
    """top_k = 1 makes every target a point mass on the argmax: the sampled
    step must reproduce the greedy step exactly, for any uniforms."""
    war, model = tiny["war"], tiny["model"]
    _, ctxs = _tiny_workload(seed=6, B=4, ctx_len=200)
    B, k = len(ctxs), 4
    pool, seq, ctx, kvs, onext, *_ = _prefill_both(tiny, ctxs)
    rng = np.random.default_rng(22)
    t = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.int32).to(DEV)
    dt = rng.integers(0, CFG.vocab, (B, k)).astype(np.int32)
    dl = [0, 2, 4, 3]
    ga, gn, sa, sn = t([0] * B), t([0] * B), t([0] * B), t([0] * B)
    war.verify_step(model, pool, seq, ctx, t(onext), t(dt), t(dl), k, ga, gn)
    war.kv_commit(pool, seq, ctx, t([-1] * B))
    u = torch.from_numpy(rng.random((B * (k + 1), 2)).astype(np.float32)).to(DEV)
    war.verify_step_sampled(model, pool, seq, ctx, t(onext), t(dt), t(dl), k, u, 1.0, 1, sa, sn)
    war.kv_commit(pool, seq, ctx, t([-1] * B))
    torch.cuda.synchronize()
    assert sa.cpu().tolist() == ga.cpu().tolist() and sn.cpu().tolist() == gn.cpu().tolist()


@pytest.mark.parametrize("mode", ["suffix", "greedy", "mixed"])
def test_verify_steps_match_oracle(tiny, mode):
    report = []
    stats = _run_steps(tiny, 3 if mode != "greedy" else 2, mode, seed={"suffix": 1, "greedy": 2, "mixed": 3}[mode],
                       report=report)
    print(f"\n[{mode}] max logit err {max(s['err'] for s in stats):.3e}; reported: {len(report)}")
    for line in report:
        print("  ", line)
    assert max(s["err"] for s in stats) < 5e-2
    # every report is a near-tie flip (gap < 0.1) or its consequence
    assert sum(s["flips"] for s in stats) >= sum(not s["same"] for s in stats)


def test_full_accept_with_decisive_lm_head():
    """LM head std x10 (top-2 gaps far above the rounding error): drafts equal
    to the oracle's greedy continuation must be accepted exactly."""
    war = _war()
    w_cpu = synth.model_weights(CFG, seed=3, norm_std=0.1, lm_std=0.2)
    W = Weights(CFG, w_cpu)
    model = war.Model(CFG, {k: v.to(DEV) for k, v in w_cpu.items()}, max_rows=64)
    tiny = {"war": war, "W": W, "model": model}
    _, ctxs = _tiny_workload(seed=4, B=4, ctx_len=200)
    pool, seq, ctx, kvs, onext, ologits, gnext, glogits = _prefill_both(tiny, ctxs)
    assert (gnext == onext).all()
    k = 5
    drafts = [greedy_decode(CFG, W, copy.deepcopy(kvs[b]), int(onext[b]), k + 1) for b in range(4)]
    dt = torch.tensor([d[:k] for d in drafts], dtype=torch.int32, device=DEV)
    acc = torch.zeros(4, dtype=torch.int32, device=DEV)
    nxt = torch.zeros(4, dtype=torch.int32, device=DEV)
    war.verify_step(model, pool, seq, ctx, torch.tensor(onext, dtype=torch.int32, device=DEV), dt,
                    None, k, acc, nxt)
    war.kv_commit(pool, seq, ctx, acc)
    assert acc.cpu().tolist() == [k] * 4
    assert nxt.cpu().tolist() == [d[k] for d in drafts]
    assert ctx.cpu().tolist() == [len(c) + k + 1 for c in ctxs]
