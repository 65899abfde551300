"""GPU parity on the 36-layer decoder's shapes (d 4096, 32 q / 8 kv heads,
head_dim 128, FFN 12288, vocab 151936).

* Reduced depth (2 layers, every width and the full vocabulary) against the
  oracle on every request: ragged draft lengths covering all three query-row
  tilings (k = 0, 2, 4, 8), contexts that are not multiples of a page or of
  an attention chunk, and the multi-chunk split-KV path.
* Prefill-append on the same shapes, then a verify step on the appended KV.
* The multi-turn append path: forked shared prefixes, an appended observation,
  then a k = 4 verify step.
* The full 36-layer workloads exactly as the benchmark runs them, checked on
  sampled requests: low load (8 x 32768 cached tokens, k = 8), high load (64
  lognormal contexts, k = 0 and k = 2) and multi-turn (forked prefixes, a
  2048-token append, then k = 4).
The cached contexts come from the seeded generator (an input of the step), so
the oracle reads the very same keys and values; after the multi-turn append
the oracle reads the cached keys and values back from the pool (the append's
own parity is checked at reduced depth).
"""
import copy

import numpy as np
import pytest
import torch

from oracle.decoder import RequestKV, Weights, forward_block
from oracle.verify import greedy_decode, prefill_request, verify_request, verify_tree_request
from paper_2607_17299_amd import harness, synth
from parity import (NEAR_TIE, compare_request, compare_tree_request, fp32_drift_tol,
                    near_sampled_decision, shared_units)

pytestmark = pytest.mark.gpu
KV_SEED = 9


def _war():
    from paper_2607_17299_amd import war
    return war


@pytest.fixture(scope="module")
def large2():
    war = _war()
    cfg = synth.reduced(synth.LARGE, 2)
    w = harness.large_weights(cfg)
    model = war.Model(cfg, w, max_rows=512)
    return {"cfg": cfg, "w": w, "model": model, "W": Weights(cfg, w), "war": war}


def _oracle_kv(cfg, seq, ctx):
    def get(l):
        a = synth.kv_context(cfg, KV_SEED, seq, l, 0, ctx, "cuda").cpu().double().numpy()
        return a[0], a[1]
    return get


def _check_step(env, st, report, tag):
    cfg, model, W = env["cfg"], env["model"], env["W"]
    pool = harness.make_pool(cfg, st.ctx_lens, st.k_max + 2)
    harness.load_contexts(pool, cfg, st.ctx_lens, st.seq_ids, KV_SEED)
    ds = harness.DeviceStep(st, with_logits=True, vocab=cfg.vocab)
    ds.verify(model, pool, logits=True)
    ds.commit(pool, discard=False)
    torch.cuda.synchronize()
    glog = ds.logits.cpu().numpy().reshape(st.B, st.k_max + 1, cfg.vocab)
    acc, nxt = ds.accept.cpu().numpy(), ds.next.cpu().numpy()
    errs = []
    for b in range(st.B):
        ctx = int(st.ctx_lens[b])
        kv = RequestKV(cfg, [_oracle_kv(cfg, int(st.seq_ids[b]), ctx)(l) for l in range(cfg.n_layers)])
        r = verify_request(cfg, W, kv, int(st.last_tokens[b]), st.drafts[b])
        errs.append(compare_request(r["logits"], glog[b], st.drafts[b], r["accept"], r["next"],
                                    int(acc[b]), int(nxt[b]), report, f"{tag} req {b}")["err"])
        # the committed KV of the new rows matches the oracle's
        keep = int(acc[b]) + 1
        g = pool.gather_kv(int(st.seq_ids[b]), ctx + keep, cfg.n_layers - 1).double().cpu().numpy()
        nk, nv = r["new_kv"][cfg.n_layers - 1]
        np.testing.assert_allclose(g[0][:, ctx:], nk[:, :keep], atol=3e-2, rtol=2e-2)
        np.testing.assert_allclose(g[1][:, ctx:], nv[:, :keep], atol=3e-2, rtol=2e-2)
    got_ctx = ds.ctx.cpu().numpy()
    np.testing.assert_array_equal(got_ctx, st.ctx_lens + acc + 1)
    return max(errs)


@pytest.mark.parametrize("k,lens,ctxs", [
    (0, [0, 0, 0], [1000, 2500, 4097]),
    (2, [2, 0, 1], [700, 3001, 1024]),
    (4, [4, 1, 3], [1500, 33, 2048]),
    (8, [8, 5, 0], [3000, 1100, 2500]),
    # 108 rows: two 64-row m-blocks, taken by one GEMM workgroup
    (8, [8, 3, 0, 8, 1, 6, 2, 8, 0, 5, 8, 4],
     [300, 1200, 77, 2100, 640, 90, 1500, 33, 1025, 400, 260, 700]),
    # 50 rows: the projections in one 64-row tile (14 padding rows)
    (4, [4, 0, 2, 4, 1, 3, 4, 0, 4, 2], [500, 17, 1600, 48, 900, 2049, 64, 311, 1200, 95]),
    # 72 and 80 rows: qkv and o in one 80-row column-quarter tile, gate/up and down in k_gemm
    (8, [8, 0, 3, 8, 5, 1, 8, 2], [900, 64, 1500, 33, 2100, 400, 17, 1025]),
    (4, [b % 5 for b in range(16)], [40 + (53 * b) % 900 for b in range(16)]),
    # 150 rows: two 80-row m-blocks in one workgroup (10 padding rows)
    (2, [b % 3 for b in range(50)], [16 + (37 * b) % 300 for b in range(50)]),
])
def test_reduced_depth_verify_matches_oracle(large2, k, lens, ctxs):
    cfg = large2["cfg"]
    B = len(ctxs)
    rng = np.random.default_rng(k)
    drafts = [rng.integers(0, cfg.vocab, n).tolist() for n in lens]
    st = harness.Step(np.arange(B, dtype=np.int32), np.array(ctxs, np.int32),
                      synth.uniform_tokens(k + 40, B, cfg.vocab), drafts, k)
    report = []
    err = _check_step(large2, st, report, f"k={k}")
    print(f"\nk={k}: max logit err {err:.3e}; reported {report}")


@pytest.mark.parametrize("k", [2, 4, 8])
def test_rows_do_not_depend_on_later_drafts(large2, k):
    """A row's result depends only on the tokens up to it: changing only the
    last draft token (the input of the last row) of one request leaves every
    earlier row's logits bitwise unchanged, for one, two and three row tiles
    and across key chunks.  (The attention's lazy rescaling is decided per row,
    so no row's rounding follows another row's rescale events.)"""
    cfg, model = large2["cfg"], large2["model"]
    ctxs = np.array([2100, 900, 4500, 3333], np.int32)
    B = len(ctxs)
    rng = np.random.default_rng(300 + k)
    last = synth.uniform_tokens(300 + k, B, cfg.vocab)
    drafts = [[int(v) for v in rng.integers(0, cfg.vocab, k)] for _ in range(B)]
    pool = harness.make_pool(cfg, ctxs, k + 2)
    harness.load_contexts(pool, cfg, ctxs, np.arange(B), KV_SEED)
    out = []
    for variant in range(2):
        d = [list(x) for x in drafts]
        if variant:
            d[1][-1] = (d[1][-1] + 12345) % cfg.vocab
        ds = harness.DeviceStep(harness.Step(np.arange(B, dtype=np.int32), ctxs, last, d, k),
                                with_logits=True, vocab=cfg.vocab)
        ds.verify(model, pool, logits=True)
        ds.commit(pool, discard=True)
        torch.cuda.synchronize()
        out.append(ds.logits.cpu().numpy().reshape(B, k + 1, cfg.vocab))
    for b in range(B):
        rows = k if b == 1 else k + 1   # request 1's last row saw the changed token
        np.testing.assert_array_equal(out[0][b, :rows], out[1][b, :rows], err_msg=f"k={k} req {b}")
    assert not np.array_equal(out[0][1, k], out[1][1, k])


@pytest.mark.parametrize("T,top_k", [(1.0, 200), (0.7, 50)])
def test_reduced_depth_sampled_matches_oracle(large2, T, top_k):
    """Sampled verification at full widths (d 4096, vocabulary 151,936; 2
    layers): ragged drafts, half of them the oracle's greedy continuation, and
    seeded uniforms.  The GPU's decisions equal the oracle's sampled rule on the
    oracle's logits with the same uniforms, except where the measured logit
    error could move a draw (reported), and the committed context lengths
    follow the GPU's accept lengths."""
    from oracle.sampling import verify_sampled
    war, cfg, model, W = large2["war"], large2["cfg"], large2["model"], large2["W"]
    ctxs = np.array([1500, 33, 2049, 700], np.int32)
    B, k = len(ctxs), 4
    rng = np.random.default_rng(int(T * 10) + top_k)
    last = synth.uniform_tokens(77 + top_k, B, cfg.vocab)
    pool = harness.make_pool(cfg, ctxs, k + 2)
    harness.load_contexts(pool, cfg, ctxs, np.arange(B), KV_SEED)
    kvs = [RequestKV(cfg, [_oracle_kv(cfg, b, int(ctxs[b]))(l) for l in range(cfg.n_layers)]) for b in range(B)]
    drafts = []
    for b in range(B):
        n = int(rng.integers(0, k + 1))
        if b % 2 == 0:
            d = greedy_decode(cfg, W, copy.deepcopy(kvs[b]), int(last[b]), n)
        else:
            d = [int(x) for x in rng.integers(0, cfg.vocab, n)]
        drafts.append(d)
    dt = np.zeros((B, k), np.int32)
    for b, d in enumerate(drafts):
        dt[b, : len(d)] = d
    u = rng.random((B * (k + 1), 2)).astype(np.float32)
    t = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.int32).to("cuda")
    seq, ctx = t(np.arange(B)), t(ctxs)
    acc, nx = t([0] * B), t([0] * B)
    logits = torch.zeros((B * (k + 1), cfg.vocab), device="cuda")
    war.verify_step_sampled(model, pool, seq, ctx, t(last), t(dt), t([len(d) for d in drafts]), k,
                            torch.from_numpy(u).to("cuda"), T, top_k, acc, nx, logits)
    torch.cuda.synchronize()
    g_acc, g_nxt = acc.cpu().numpy(), nx.cpu().numpy()
    glog = logits.cpu().numpy().reshape(B, k + 1, cfg.vocab)
    report, exact = [], 0
    for b in range(B):
        n = len(drafts[b])
        r = verify_request(cfg, W, kvs[b], int(last[b]), drafts[b])
        uu = u[b * (k + 1): b * (k + 1) + n + 1].astype(np.float64)
        rs = verify_sampled(r["logits"], drafts[b], uu[:, 0], uu[:, 1], T, top_k)
        err = float(np.abs(glog[b, : n + 1] - r["logits"]).max())
        assert err < 5e-2, (b, err)
        assert 0 <= g_acc[b] <= n and 0 <= g_nxt[b] < cfg.vocab
        if (int(g_acc[b]), int(g_nxt[b])) != (rs["accept"], rs["next"]):
            assert near_sampled_decision(r["logits"], T, top_k, err, rs["margins"]), \
                (b, (int(g_acc[b]), int(g_nxt[b])), (rs["accept"], rs["next"]), rs["margins"], err)
            report.append(f"req {b}: near-boundary sample differs")
        else:
            exact += 1
    war.kv_commit(pool, seq, ctx, acc)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ctx.cpu().numpy(), ctxs + g_acc + 1)
    print(f"\nsampled at full widths T={T} top_k={top_k}: accept {g_acc.tolist()}, {exact} exact, "
          f"reported {report}")


@pytest.mark.parametrize("k", [3, 11])
def test_reduced_depth_tree_matches_oracle(large2, k):
    """Tree drafts on the 36-layer shapes (2 layers): random trees of ragged
    sizes (k = 11 fills the 48-row attention block), contexts across several
    key chunks and off page boundaries.  Node logits, accepted path, next
    token; after the commit the last layer's cache of the new slots is the
    accepted path's KV."""
    cfg, model, W = large2["cfg"], large2["model"], large2["W"]
    ctxs = [1500, 3001, 2048, 77]
    B = len(ctxs)
    rng = np.random.default_rng(100 + k)
    sizes = [k, int(rng.integers(1, k + 1)), 0, k]
    drafts = [rng.integers(0, cfg.vocab, n).tolist() for n in sizes]
    parents = [[int(rng.integers(0, i + 1)) for i in range(n)] for n in sizes]
    st = harness.Step(np.arange(B, dtype=np.int32), np.array(ctxs, np.int32),
                      synth.uniform_tokens(k + 90, B, cfg.vocab), drafts, k, parents)
    pool = harness.make_pool(cfg, st.ctx_lens, k + 2)
    harness.load_contexts(pool, cfg, st.ctx_lens, st.seq_ids, KV_SEED)
    ds = harness.DeviceStep(st, with_logits=True, vocab=cfg.vocab)
    ds.verify_tree(model, pool, logits=True)
    ds.commit(pool, discard=False)
    torch.cuda.synchronize()
    glog = ds.logits.cpu().numpy().reshape(B, k + 1, cfg.vocab)
    acc, nxt, path = ds.accept.cpu().numpy(), ds.next.cpu().numpy(), ds.path.cpu().numpy()
    report = []
    for b in range(B):
        tag = f"k={k} req {b}"
        kv = RequestKV(cfg, [_oracle_kv(cfg, b, ctxs[b])(l) for l in range(cfg.n_layers)])
        r = verify_tree_request(cfg, W, kv, int(st.last_tokens[b]), drafts[b], parents[b])
        a = int(acc[b])
        same = compare_tree_request(r, glog[b], [int(st.last_tokens[b])] + drafts[b], parents[b], a,
                                    int(nxt[b]), path[b, :a], report, tag)
        if same:
            g = pool.gather_kv(b, ctxs[b] + a + 1, cfg.n_layers - 1).double().cpu().numpy()
            nk, nv = r["new_kv"][cfg.n_layers - 1]
            np.testing.assert_allclose(g[0][:, ctxs[b]:], nk, atol=3e-2, rtol=2e-2, err_msg=tag)
            np.testing.assert_allclose(g[1][:, ctxs[b]:], nv, atol=3e-2, rtol=2e-2, err_msg=tag)
    np.testing.assert_array_equal(ds.ctx.cpu().numpy(), st.ctx_lens + acc + 1)
    print(f"\ntree k={k}: reported {report}")


def test_reduced_depth_tree_greedy_branch_accepted(large2):
    """A tree holding the target's greedy continuation on one branch, under
    distractor branches (decisive LM head): the GPU accepts exactly that
    branch, and the emitted tokens are the greedy stream."""
    war, cfg = large2["war"], large2["cfg"]
    w = harness.large_weights(cfg, lm_std=0.2)
    model = war.Model(cfg, w, max_rows=64)
    W = Weights(cfg, w)
    ctxs = np.array([1200, 2000], np.int32)
    last = synth.uniform_tokens(62, 2, cfg.vocab)
    rng = np.random.default_rng(62)
    drafts, parents, conts = [], [], []
    for b in range(2):
        kv = RequestKV(cfg, [_oracle_kv(cfg, b, int(ctxs[b]))(l) for l in range(cfg.n_layers)])
        g = greedy_decode(cfg, W, kv, int(last[b]), 5)
        x = [int(v) for v in rng.integers(0, cfg.vocab, 4)]
        # greedy branch 2 -> 3 -> 6 -> 8; distractors 1, 4, 5, 7
        drafts.append([x[0], g[0], g[1], x[1], x[2], g[2], x[3], g[3]])
        parents.append([0, 0, 2, 2, 1, 3, 6, 6])
        conts.append(g)
    st = harness.Step(np.arange(2, dtype=np.int32), ctxs, last, drafts, 8, parents)
    pool = harness.make_pool(cfg, st.ctx_lens, 10)
    harness.load_contexts(pool, cfg, st.ctx_lens, st.seq_ids, KV_SEED)
    ds = harness.DeviceStep(st)
    ds.verify_tree(model, pool)
    ds.commit(pool, discard=False)
    assert ds.accept.cpu().tolist() == [4, 4]
    assert ds.path.cpu().numpy()[:, :4].tolist() == [[2, 3, 6, 8]] * 2
    assert ds.next.cpu().tolist() == [c[4] for c in conts]


def test_reduced_depth_sibling_drafts_accepted(large2):
    """Drafts = the oracle's own greedy continuation (decisive LM head) are
    accepted in full on the GPU."""
    war = large2["war"]
    cfg = large2["cfg"]
    w = harness.large_weights(cfg, lm_std=0.2)
    model = war.Model(cfg, w, max_rows=64)
    W = Weights(cfg, w)
    ctxs = np.array([1200, 2000], np.int32)
    last = synth.uniform_tokens(61, 2, cfg.vocab)
    k = 4
    drafts = []
    for b in range(2):
        kv = RequestKV(cfg, [_oracle_kv(cfg, b, int(ctxs[b]))(l) for l in range(cfg.n_layers)])
        toks, x = [], int(last[b])
        for _ in range(k + 1):
            r = verify_request(cfg, W, kv, x, [])
            kv.append(r["new_kv"], 1)
            x = r["next"]
            toks.append(x)
        drafts.append(toks)
    st = harness.Step(np.arange(2, dtype=np.int32), ctxs, last, [d[:k] for d in drafts], k)
    pool = harness.make_pool(cfg, st.ctx_lens, k + 2)
    harness.load_contexts(pool, cfg, st.ctx_lens, st.seq_ids, KV_SEED)
    ds = harness.DeviceStep(st)
    ds.verify(model, pool)
    ds.commit(pool, discard=False)
    assert ds.accept.cpu().tolist() == [k, k]
    assert ds.next.cpu().tolist() == [d[k] for d in drafts]


@pytest.mark.parametrize("ctxs,n_new", [([512, 96], [300, 45]), ([77, 4000], [1, 33]), ([1024, 333], [64, 129])])
def test_reduced_depth_prefill_append(large2, ctxs, n_new):
    """war_prefill_append at full widths (2 layers): the last row's logits and
    next token, and the appended K/V, against the oracle.  Lengths cover one
    token, a 32-token row block plus one (the prefill attention's row blocks
    hold 32 tokens x 4 query heads), exact multiples, several row blocks, and
    contexts that end inside a page."""
    war, cfg, model, W = large2["war"], large2["cfg"], large2["model"], large2["W"]
    ctxs = np.array(ctxs, np.int32)
    pool = harness.make_pool(cfg, ctxs + np.array(n_new), 8)
    harness.load_contexts(pool, cfg, ctxs, [0, 1], KV_SEED)
    toks = [synth.uniform_tokens(70 + b, n, cfg.vocab) for b, n in enumerate(n_new)]
    t = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.int32).cuda()
    ctx_d = t(ctxs)
    nxt = t([0, 0])
    last = torch.zeros((2, cfg.vocab), device="cuda")
    war.prefill_append(model, pool, t([0, 1]), ctx_d, n_new, t(np.concatenate(toks)), nxt, last)
    assert ctx_d.cpu().tolist() == (ctxs + np.array(n_new)).tolist()
    gl = last.cpu().numpy()
    for b in range(2):
        kv = RequestKV(cfg, [_oracle_kv(cfg, b, int(ctxs[b]))(l) for l in range(cfg.n_layers)])
        r = prefill_request(cfg, W, kv, toks[b])
        err = np.abs(gl[b] - r["logits"][-1]).max()
        assert err < 5e-2, err
        if int(nxt[b]) != r["next"]:
            s = np.sort(r["logits"][-1])
            assert s[-1] - s[-2] < NEAR_TIE and s[-1] - s[-2] <= 2 * err, (b, s[-1] - s[-2], err)
        g = pool.gather_kv(b, int(ctxs[b]) + n_new[b], 1).double().cpu().numpy()
        K, V = kv.get(1)
        np.testing.assert_allclose(g[0][:, ctxs[b]:], K[:, ctxs[b]:], atol=3e-2, rtol=2e-2)
        np.testing.assert_allclose(g[1][:, ctxs[b]:], V[:, ctxs[b]:], atol=3e-2, rtol=2e-2)


@pytest.mark.parametrize("prefix", [256, 2048])
def test_reduced_depth_multi_turn(large2, prefix):
    """The multi-turn append path on the full widths at 2 layers: 2 groups x 2
    trajectories whose cached contexts share a forked prefix (256 tokens: less
    than an attention chunk; 2048: two whole chunks, attended once per sibling
    pair) plus 200 private tokens (not a page multiple), a 300-token
    observation appended to each (prefill chunks span the 512-row workspace),
    then one k = 4 verify step.  Trajectory 0 drafts the oracle's own greedy
    continuation (all accepted), trajectory 1 the same with its second draft
    replaced (one accepted), the others draft from the suffix drafter."""
    war, cfg, model, W = large2["war"], large2["cfg"], large2["model"], large2["W"]
    mt = harness.multi_turn_inputs(seed=11, groups=2, per_group=2, prefix=prefix, private=200,
                                   n_new=300, vocab=cfg.vocab)
    pool = harness.multi_turn_pool(cfg, mt, 4)
    harness.load_multi_turn(pool, cfg, mt, KV_SEED)
    bt = pool.block_tables.cpu().numpy()
    npg = prefix // 16
    np.testing.assert_array_equal(bt[0, :npg], bt[1, :npg])      # the prefix pages are shared
    np.testing.assert_array_equal(bt[2, :npg], bt[3, :npg])
    assert len(set(bt[0, npg:npg + 13]) & set(bt[1, npg:npg + 13])) == 0   # the private ones are not
    nxt, ctx_d, last = harness.multi_turn_append(model, pool, mt, last_logits=True)
    torch.cuda.synchronize()
    assert ctx_d.cpu().tolist() == [mt.cached + mt.n_new] * mt.n
    gl, gnext = last.cpu().numpy(), nxt.cpu().numpy()
    kvs, conts, onext = [], [], []
    for s in range(mt.n):
        full = [harness.multi_turn_kv(cfg, mt, KV_SEED, s, l).cpu().double().numpy() for l in range(cfg.n_layers)]
        kv = RequestKV(cfg, [(a[0], a[1]) for a in full])
        hf, new_kv = forward_block(cfg, W, [int(t) for t in mt.obs[s]], kv.length, kv.get, want_logits=False)
        kv.append(new_kv, mt.n_new)
        z = hf[-1] @ W.get("w_lm").T
        err = np.abs(gl[s] - z).max()
        assert err < 5e-2, (s, err)
        g = int(np.argmax(z))
        if int(gnext[s]) != g:
            zs = np.sort(z)
            assert zs[-1] - zs[-2] <= 2 * err, (s, gnext[s], g)
        # the appended keys/values in the pages match the oracle's
        got = pool.gather_kv(s, mt.cached + mt.n_new, cfg.n_layers - 1).double().cpu().numpy()
        K, V = kv.get(cfg.n_layers - 1)
        np.testing.assert_allclose(got[0][:, mt.cached:], K[:, mt.cached:], atol=3e-2, rtol=2e-2)
        np.testing.assert_allclose(got[1][:, mt.cached:], V[:, mt.cached:], atol=3e-2, rtol=2e-2)
        np.testing.assert_array_equal(got[0][:, :mt.cached], full[-1][0])   # cached part untouched
        kvs.append(kv)
        onext.append(g)
        conts.append(greedy_decode(cfg, W, RequestKV(cfg, list(kv.layers)), g, 4))
    # the verify step's pending tokens are the oracle's argmax after the append
    onext = np.array(onext, np.int32)
    base = harness.multi_turn_step(mt, onext, 4)
    drafts = [conts[0], [conts[1][0], (conts[1][1] + 1) % cfg.vocab] + conts[1][2:]] + base.drafts[2:]
    st = harness.Step(mt.seq_ids, base.ctx_lens, onext, drafts, 4)
    ds = harness.DeviceStep(st, with_logits=True, vocab=cfg.vocab)
    ds.verify(model, pool, logits=True)
    torch.cuda.synchronize()
    n_items = war.debug_workspace(model, "n_items", torch.int32, (2,)).cpu().tolist()
    # 2048 shared tokens = 2 chunks of 1024: attended once per run of siblings
    # whose live rows fit one 32-row block together
    runs = [shared_units([4 * (len(d) + 1) for d in st.drafts[g:g + 2]], 32) for g in (0, 2)]
    saved = sum(2 * (2 - len(r)) for r in runs) if prefix == 2048 else 0
    assert n_items == [n_items[0], n_items[0] - saved], (n_items, runs)
    print(f"shared-prefix runs {runs}: {saved} units saved")
    ds.commit(pool, discard=False)
    torch.cuda.synchronize()
    glog = ds.logits.cpu().numpy().reshape(st.B, 5, cfg.vocab)
    acc, nx = ds.accept.cpu().numpy(), ds.next.cpu().numpy()
    report, o_acc = [], []
    for s in range(mt.n):
        r = verify_request(cfg, W, kvs[s], int(onext[s]), st.drafts[s])
        compare_request(r["logits"], glog[s], st.drafts[s], r["accept"], r["next"], int(acc[s]), int(nx[s]),
                        report, f"multi_turn traj {s}")
        o_acc.append(r["accept"])
    # losslessness on the oracle side: its own continuation is accepted in full
    assert o_acc[0] == 4 and o_acc[1] == 1, o_acc
    np.testing.assert_array_equal(ds.ctx.cpu().numpy(), st.ctx_lens + acc + 1)
    print(f"\nmulti_turn: accept {acc.tolist()}; {report}")


# The full-size checks spend minutes in the oracle's float64 forward on the
# host (36 layers, weights widened layer by layer); it prints each layer it
# reaches, so a longer per-test limit than the GPU steps' still ends a hang.
ORACLE_SLOW = pytest.mark.timeout(420)


def _oracle_kv_stream(cfg, kv_seed, seq, ctx, tag):
    """Layer-by-layer cached K/V of one request from the seeded generator."""
    cache = {}

    def kv_get(l):
        if l not in cache:
            print(f"{tag}: oracle layer {l}", flush=True)   # progress: the oracle takes minutes
            a = synth.kv_context(cfg, kv_seed, seq, l, 0, ctx, "cuda").cpu().double().numpy()
            cache.clear()
            cache[l] = (a[0], a[1])
        return cache[l]
    return kv_get


def _full_size_check(st, kv_seed, sample, tag, setup=None, chunk=None):
    """Run one verify step of the 36-layer model on the GPU with logits and
    recompute the sampled requests with the oracle (float64, and its fp32-
    accumulation mode for the tolerance), layer by layer.  `setup`, when given,
    builds (model, pool, step, kv_get factory) instead of the seeded contexts.
    `chunk`, when given, is the attention chunk length the step must have used
    (the step setup picks 1024 or 2048 keys per item)."""
    war = _war()
    cfg = synth.LARGE
    w = harness.large_weights(cfg)
    if setup is None:
        model = war.Model(cfg, w, max_rows=1024)
        pool = harness.make_pool(cfg, st.ctx_lens, max(st.k_max, 2) + 8)
        harness.load_contexts(pool, cfg, st.ctx_lens, st.seq_ids, kv_seed)
        kv_source = lambda b, ctx: _oracle_kv_stream(cfg, kv_seed, int(st.seq_ids[b]), ctx, f"{tag} req {b}")
    else:
        model, pool, st, kv_source = setup(war, cfg, w)
    ds = harness.DeviceStep(st, with_logits=True, vocab=cfg.vocab)
    ds.verify(model, pool, logits=True)
    torch.cuda.synchronize()
    if chunk is not None:
        n_items = war.debug_workspace(model, "n_items", torch.int32, (4,)).cpu().tolist()
        assert n_items[3] == chunk, (tag, n_items)
    ds.commit(pool, discard=False)
    torch.cuda.synchronize()
    glog = ds.logits.cpu().numpy().reshape(st.B, st.k_max + 1, cfg.vocab)
    acc, nxt = ds.accept.cpu().numpy(), ds.next.cpu().numpy()
    np.testing.assert_array_equal(ds.ctx.cpu().numpy(), st.ctx_lens + acc + 1)
    W = Weights(cfg, w, cache=False)
    from oracle.accept import accept_length, argmax_lowest
    report, out = [], []
    for b in sample:
        ctx = int(st.ctx_lens[b])
        kv_get = kv_source(b, ctx)
        tokens = [int(st.last_tokens[b])] + list(st.drafts[b])
        o64, _ = forward_block(cfg, W, tokens, ctx, kv_get)
        o32, _ = forward_block(cfg, W, tokens, ctx, kv_get, precision="fp32")
        tol = fp32_drift_tol(o64, o32)
        g = argmax_lowest(o64)
        a = accept_length(st.drafts[b], g)
        s = compare_request(o64, glog[b], st.drafts[b], a, int(g[a]), int(acc[b]), int(nxt[b]),
                            report, f"{tag} req {b}", tol=tol)
        out.append((b, round(s["err"], 4), round(tol, 4), a))
    print(f"\n{tag}: (request, max logit err, bound, oracle accept) {out}; GPU accept {acc.tolist()}; {report}")


@ORACLE_SLOW
def test_full_size_low_load_sampled():
    """The benchmark's workload at full size (36 layers, 8 x 32768, k = 8);
    requests 0 and 7 are recomputed by the oracle.  The batch has enough keys
    for 2048-key attention chunks (8 x 17 items), so those are what it checks."""
    _full_size_check(harness.low_load_step(), 5, [0, 7], "low_load", chunk=2048)


@ORACLE_SLOW
def test_full_size_high_load_sampled():
    """64 requests with lognormal contexts and k = 0 (plain batched decode);
    the shortest, the median and the longest request are recomputed by the
    oracle."""
    st = harness.high_load_step(k=0)
    order = np.argsort(st.ctx_lens, kind="stable")
    sample = [int(order[0]), int(order[len(order) // 2]), int(order[-1])]
    _full_size_check(st, 5, sample, "high_load")


@ORACLE_SLOW
def test_full_size_multi_turn_sampled():
    """16 trajectories in 4 groups sharing a forked 8192-token prefix (24576
    cached tokens each), a 2048-token observation appended to each with
    war_prefill_append, then the k = 4 verify step (shared-prefix attention
    units).  Trajectories 0 and 5 (two groups) are recomputed by the oracle
    from the cached keys and values the pool holds after the append."""
    def setup(war, cfg, w):
        model = war.Model(cfg, w, max_rows=2048)    # the benchmark's prefill chunk rows
        mt = harness.multi_turn_inputs(vocab=cfg.vocab)
        pool = harness.multi_turn_pool(cfg, mt, 4)
        harness.load_multi_turn(pool, cfg, mt, 5)
        nxt, ctx_dev, _ = harness.multi_turn_append(model, pool, mt)
        torch.cuda.synchronize()
        assert ctx_dev.cpu().tolist() == [mt.cached + mt.n_new] * mt.n
        st = harness.multi_turn_step(mt, nxt.cpu().numpy(), 4)

        def kv_source(b, ctx):
            cache = {}

            def kv_get(l):
                if l not in cache:
                    print(f"multi_turn traj {b}: oracle layer {l}", flush=True)
                    a = pool.gather_kv(int(st.seq_ids[b]), ctx, l).cpu().double().numpy()
                    cache.clear()
                    cache[l] = (a[0], a[1])
                return cache[l]
            return kv_get
        return model, pool, st, kv_source
    # forked siblings keep 1024-key chunks (shared chunks read together hit L2)
    _full_size_check(None, 5, [0, 5], "multi_turn", setup=setup, chunk=1024)


@ORACLE_SLOW
def test_full_size_high_load_k2_sampled():
    """64 requests with lognormal contexts and k = 2.  The shortest and the
    longest request draft the oracle's own greedy continuation with ~30% of the
    positions corrupted (acceptance and rollback both exercised); the other
    requests draft random tokens.  The two are recomputed by the oracle."""
    from oracle.accept import argmax_lowest
    cfg = synth.LARGE
    st = harness.high_load_step(k=0)
    sample = [int(np.argmin(st.ctx_lens)), int(np.argmax(st.ctx_lens))]
    W = Weights(cfg, harness.large_weights(cfg), cache=False)
    rng = np.random.default_rng(12)
    drafts = [rng.integers(0, cfg.vocab, 2).tolist() for _ in range(st.B)]
    cont = []
    for b in sample:
        kv_get = _oracle_kv_stream(cfg, 5, b, int(st.ctx_lens[b]), f"teacher req {b}")
        x = int(st.last_tokens[b])
        z, _ = forward_block(cfg, W, [x], int(st.ctx_lens[b]), kv_get)
        g0 = int(argmax_lowest(z)[0])
        z, _ = forward_block(cfg, W, [x, g0], int(st.ctx_lens[b]), kv_get)
        cont.append([g0, int(argmax_lowest(z)[1])])
    del W
    for b, d in zip(sample, harness.corrupt(cont, 0.3, seed=4, vocab=cfg.vocab)):
        drafts[b] = d
    st = harness.Step(st.seq_ids, st.ctx_lens, st.last_tokens, drafts, 2)
    _full_size_check(st, 5, sample, "high_load_k2")


@ORACLE_SLOW
def test_full_size_tree_sampled():
    """Tree drafts at full depth (36 layers, full widths): 4 requests over
    seeded contexts with 4-node trees.  Request 0's root has the oracle's own
    greedy token as its second child (with a grandchild), so the GPU must
    accept that branch; request 2 carries a random tree.  Both are recomputed
    by the oracle node by node (every node's root path decoded as a chain),
    with the bound from the fp32 drift of the deepest path; request 0's
    committed cache (last layer) must be the accepted path's K/V."""
    war = _war()
    cfg = synth.LARGE
    w = harness.large_weights(cfg)
    model = war.Model(cfg, w, max_rows=64)
    W = Weights(cfg, w, cache=True)
    kv_seed = 5
    ctxs = np.array([3000, 4500, 1200, 6000], np.int32)
    B = len(ctxs)
    last = synth.uniform_tokens(70, B, cfg.vocab)
    rng = np.random.default_rng(70)

    def kv_of(b):
        layers = []
        for l in range(cfg.n_layers):
            a = synth.kv_context(cfg, kv_seed, b, l, 0, int(ctxs[b]), "cuda").cpu().double().numpy()
            layers.append((a[0], a[1]))
        return RequestKV(cfg, layers)
    kv0 = kv_of(0)
    z, _ = forward_block(cfg, W, [int(last[0])], int(ctxs[0]), kv0.get)
    from oracle.accept import argmax_lowest
    g0 = int(argmax_lowest(z)[0])
    rnd = [[int(v) for v in rng.integers(0, cfg.vocab, 4)] for _ in range(B)]
    drafts = [[rnd[0][0], g0, rnd[0][1], rnd[0][2]], rnd[1], rnd[2], rnd[3]]
    parents = [[0, 0, 2, 1], [0, 1, 1, 0], [0, 1, 1, 0], [0, 0, 0, 0]]
    st = harness.Step(np.arange(B, dtype=np.int32), ctxs, last, drafts, 4, parents)
    pool = harness.make_pool(cfg, st.ctx_lens, 6)
    harness.load_contexts(pool, cfg, st.ctx_lens, st.seq_ids, kv_seed)
    ds = harness.DeviceStep(st, with_logits=True, vocab=cfg.vocab)
    ds.verify_tree(model, pool, logits=True)
    ds.commit(pool, discard=False)
    torch.cuda.synchronize()
    glog = ds.logits.cpu().numpy().reshape(B, 5, cfg.vocab)
    acc, nxt, path = ds.accept.cpu().numpy(), ds.next.cpu().numpy(), ds.path.cpu().numpy()
    np.testing.assert_array_equal(ds.ctx.cpu().numpy(), st.ctx_lens + acc + 1)
    report, out = [], []
    for b, kv in ((0, kv0), (2, kv_of(2))):
        tag = f"full-size tree req {b}"
        r = verify_tree_request(cfg, W, kv, int(last[b]), drafts[b], parents[b])
        # the deepest root path: nodes 2, 3 (request 0) or 1, 2 (request 2)
        deep = [int(last[b])] + ([drafts[b][1], drafts[b][2]] if b == 0 else [drafts[b][0], drafts[b][1]])
        o64, kv64 = forward_block(cfg, W, deep, int(ctxs[b]), kv.get)
        o32, kv32 = forward_block(cfg, W, deep, int(ctxs[b]), kv.get, precision="fp32")
        tol = fp32_drift_tol(o64, o32)
        L = cfg.n_layers - 1
        kv_tol = max(3e-2, 1.5 * max(float(np.abs(kv64[L][i] - kv32[L][i]).max()) for i in (0, 1)))
        a = int(acc[b])
        same = compare_tree_request(r, glog[b], [int(last[b])] + drafts[b], parents[b], a, int(nxt[b]),
                                    path[b, :a], report, tag, tol=tol)
        out.append((b, a, [int(x) for x in path[b, :a]], round(tol, 4), round(kv_tol, 4)))
        if b == 0:
            # the planted greedy child is accepted unless the root is a near-tie
            assert a >= 1 or report, (tag, a)
        if same:
            g = pool.gather_kv(b, int(ctxs[b]) + a + 1, L).double().cpu().numpy()
            nk, nv = r["new_kv"][L]
            np.testing.assert_allclose(g[0][:, ctxs[b]:], nk, atol=kv_tol, err_msg=tag)
            np.testing.assert_allclose(g[1][:, ctxs[b]:], nv, atol=kv_tol, err_msg=tag)
    print(f"\nfull-size tree: (request, GPU accept, path, logit bound, kv bound) {out}; {report}")


@ORACLE_SLOW
def test_full_size_prefill_append():
    """The append at full depth: two trajectories with 4000 and 4111 cached
    tokens (seeded keys and values) each receive 64 new tokens through
    war_prefill_append (36 layers).  The last row's logits and next token, and
    the appended keys and values of the first, a middle and the last layer,
    are compared with the oracle's float64 forward over the same 64 tokens.
    The logit bound is max(5e-2, 1.5 x the drift of the oracle's fp32-
    accumulation mode), measured on trajectory 0 (the KV bound likewise, never
    below 3e-2)."""
    from oracle.accept import argmax_lowest, top2_gap
    from parity import NEAR_TIE
    war = _war()
    cfg = synth.LARGE
    w = harness.large_weights(cfg)
    model = war.Model(cfg, w, max_rows=2048)
    ctxs = np.array([4000, 4111], np.int32)
    n_new = [64, 64]
    kv_seed = 5
    pool = harness.make_pool(cfg, ctxs + 64, 8)
    harness.load_contexts(pool, cfg, ctxs, [0, 1], kv_seed)
    toks = [synth.uniform_tokens(80 + b, 64, cfg.vocab) for b in range(2)]
    t = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.int32).cuda()
    ctx_d, nxt = t(ctxs), t([0, 0])
    last = torch.zeros((2, cfg.vocab), device="cuda")
    war.prefill_append(model, pool, t([0, 1]), ctx_d, n_new, t(np.concatenate(toks)), nxt, last)
    torch.cuda.synchronize()
    assert ctx_d.cpu().tolist() == (ctxs + 64).tolist()
    gl, gn = last.cpu().numpy(), nxt.cpu().numpy()
    W = Weights(cfg, w, cache=False)
    layers = (0, 17, 35)
    got = {(b, l): pool.gather_kv(b, int(ctxs[b]) + 64, l)[:, :, int(ctxs[b]):].double().cpu().numpy()
           for b in range(2) for l in layers}
    tol = kv_tol = None
    report, out = [], []
    for b in range(2):
        kv_get = _oracle_kv_stream(cfg, kv_seed, b, int(ctxs[b]), f"append traj {b}")
        o64, kv64 = forward_block(cfg, W, [int(x) for x in toks[b]], int(ctxs[b]), kv_get)
        if tol is None:
            o32, kv32 = forward_block(cfg, W, [int(x) for x in toks[b]], int(ctxs[b]), kv_get, precision="fp32")
            tol = fp32_drift_tol(o64[-1:], o32[-1:])
            kv_tol = max(3e-2, 1.5 * max(float(np.abs(kv64[l][i] - kv32[l][i]).max())
                                         for l in layers for i in (0, 1)))
        err = float(np.abs(gl[b] - o64[-1]).max())
        assert err <= tol, (b, err, tol)
        g = int(argmax_lowest(o64[-1:])[0])
        if int(gn[b]) != g:
            gap = float(top2_gap(o64[-1:])[0])
            assert gap < NEAR_TIE, (b, int(gn[b]), g, gap)
            report.append(f"traj {b}: next {int(gn[b])} vs {g} at gap {gap:.3g}")
        kv_err = 0.0
        for l in layers:
            for i in (0, 1):
                e = float(np.abs(got[(b, l)][i] - kv64[l][i]).max())
                assert e <= kv_tol, (b, l, i, e, kv_tol)
                kv_err = max(kv_err, e)
        out.append((b, round(err, 4), round(tol, 4), round(kv_err, 4), round(kv_tol, 4)))
    print(f"\nappend at full depth: (traj, logit err, bound, kv err, kv bound) {out}; {report}")
