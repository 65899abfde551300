"""GPU edge cases on the tiny decoder (2 layers, 4/2 heads, vocab 4096):

* the largest batch a step takes (1024 requests), with contexts of 0 tokens and
  of every length around the 16-token page boundaries, after a prefill-append
  of all the non-empty ones in one call;
* the longest draft chain the attention row block holds (2 query heads per
  kv-head: k_max = 23, 48 rows per request), and the refusal of one more.

Pool bookkeeping is compared bit for bit with the oracle pool after the
append, the reserve, and the commit.  Logits, accept lengths and next tokens
are compared with the oracle decoder on a fixed sample of the requests that
holds every context length of the batch (the oracle takes a few seconds per
hundred requests)."""
import copy

import numpy as np
import pytest
import torch

from oracle.decoder import RequestKV, Weights
from oracle.pages import PagePool
from oracle.verify import commit_request, greedy_decode, prefill_request, verify_request
from paper_2607_17299_amd import synth
from parity import compare_request

pytestmark = pytest.mark.gpu
CFG = synth.TINY
DEV = "cuda"


@pytest.fixture(scope="module")
def tiny_wide():
    from paper_2607_17299_amd import war
    w_cpu = synth.model_weights(CFG, seed=0, norm_std=0.1)
    model = war.Model(CFG, {k: v.to(DEV) for k, v in w_cpu.items()}, max_rows=3072)
    return {"war": war, "W": Weights(CFG, w_cpu), "model": model}


def _t(a):
    return torch.as_tensor(np.asarray(a, dtype=np.int32)).to(DEV)


def _same_pool(pool, ora, tag):
    st = pool.state()
    assert st["status"] == 0, tag
    o = ora.snapshot()
    for k in ("stack", "refcount", "held", "base", "table"):
        np.testing.assert_array_equal(st[k], o[k], err_msg=f"{tag}: {k}")


def test_largest_batch_with_empty_and_page_boundary_contexts(tiny_wide):
    war, model, W = tiny_wide["war"], tiny_wide["model"], tiny_wide["W"]
    B, k, P = 1024, 2, CFG.page_size
    lens = [b % 41 for b in range(B)]                      # 0 .. 40: 0, 1, 15-17, 31-33
    ctxs = [synth.uniform_tokens(5000 + b, L, CFG.vocab) for b, L in enumerate(lens)]
    NP, MP = 4096, 8
    pool = war.Pool(CFG, NP, B, MP)
    ora = PagePool(NP, P, B, MP)

    # one append of every non-empty context (about 20k rows, several row chunks)
    ids = [b for b in range(B) if lens[b] > 0]
    ctx_a = _t([0] * len(ids))
    nxt_a = _t([0] * len(ids))
    war.prefill_append(model, pool, _t(ids), ctx_a, [lens[b] for b in ids],
                       _t(np.concatenate([ctxs[b] for b in ids])), nxt_a)
    ora.prefill_reserve(ids, [0] * len(ids), [lens[b] for b in ids])
    torch.cuda.synchronize()
    _same_pool(pool, ora, "after the append")
    assert ctx_a.cpu().tolist() == [lens[b] for b in ids]
    g_next = dict(zip(ids, nxt_a.cpu().tolist()))

    # the oracle's side: every length 0..40 at least twice, plus the first and last request
    sample = sorted(set(range(0, 82)) | {B - 1, B - 2, 512})
    rng = np.random.default_rng(41)
    kvs, pending, report = {}, [], []
    for b in range(B):
        if b in sample:
            kvs[b] = RequestKV(CFG)
            if lens[b]:
                r = prefill_request(CFG, W, kvs[b], ctxs[b])
                assert g_next[b] == r["next"] or (r["logits"][-1].max() - np.sort(r["logits"][-1])[-2]) < 0.1, \
                    f"prefill next of request {b}"
                pending.append(r["next"])
            else:
                pending.append(int(rng.integers(CFG.vocab)))
        else:
            pending.append(g_next[b] if lens[b] else int(rng.integers(CFG.vocab)))

    # drafts: the oracle's greedy continuation for a third of the sample, random otherwise
    drafts = []
    for b in range(B):
        n = int(rng.integers(0, k + 1))
        if b in sample and b % 3 == 0:
            d = greedy_decode(CFG, W, copy.deepcopy(kvs[b]), pending[b], n)
        else:
            d = [int(x) for x in rng.integers(0, CFG.vocab, n)]
        drafts.append(d)
    dl = [len(d) for d in drafts]
    dt = np.zeros((B, k), np.int32)
    for b, d in enumerate(drafts):
        dt[b, : len(d)] = d

    seq = _t(range(B))
    ctx = _t(lens)
    acc, nxt = _t([0] * B), _t([0] * B)
    logits = torch.full((B * (k + 1), CFG.vocab), float("nan"), device=DEV)
    war.verify_step(model, pool, seq, ctx, _t(pending), _t(dt), _t(dl), k, acc, nxt, logits)
    ora.reserve(list(range(B)), lens, dl)
    torch.cuda.synchronize()
    _same_pool(pool, ora, "after the reserve")
    g_acc, g_nxt = acc.cpu().numpy(), nxt.cpu().numpy()
    glog = logits.cpu().numpy().reshape(B, k + 1, CFG.vocab)
    for b in sample:
        r = verify_request(CFG, W, kvs[b], pending[b], drafts[b])
        compare_request(r["logits"], glog[b], drafts[b], r["accept"], r["next"],
                        int(g_acc[b]), int(g_nxt[b]), report, f"request {b} (ctx {lens[b]})")
        commit_request(kvs[b], r, int(g_acc[b]))
    assert all((0 <= g_acc) & (g_acc <= np.array(dl)))
    war.kv_commit(pool, seq, ctx, acc)
    new = ora.commit(list(range(B)), lens, g_acc.tolist())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ctx.cpu().numpy(), new)
    _same_pool(pool, ora, "after the commit")
    ora.check_invariants()
    # the KV the step kept (pending token and accepted drafts) reads back as the oracle's
    for b in sample:
        if kvs[b].length == 0:
            continue
        for l in range(CFG.n_layers):
            g = pool.gather_kv(b, kvs[b].length, l).double().cpu().numpy()
            K, V = kvs[b].get(l)
            np.testing.assert_allclose(g[0], K, atol=2e-2, rtol=2e-2, err_msg=f"request {b} layer {l} K")
            np.testing.assert_allclose(g[1], V, atol=2e-2, rtol=2e-2, err_msg=f"request {b} layer {l} V")
    print(f"\n1024-request step: {int((g_acc > 0).sum())} requests accepted drafts; reported: {len(report)}")
    for line in report:
        print("  ", line)


def test_longest_draft_chain(tiny_wide):
    war, model, W = tiny_wide["war"], tiny_wide["model"], tiny_wide["W"]
    G = CFG.n_q_heads // CFG.n_kv_heads
    k = 48 // G - 1                                          # 23: 48 rows per request
    lens = [100, 16, 0]
    B = len(lens)
    ctxs = [synth.uniform_tokens(7000 + b, L, CFG.vocab) for b, L in enumerate(lens)]
    pool = war.Pool(CFG, 64, B, 16)
    ids = [b for b in range(B) if lens[b]]
    ctx_a, nxt_a = _t([0] * len(ids)), _t([0] * len(ids))
    war.prefill_append(model, pool, _t(ids), ctx_a, [lens[b] for b in ids],
                       _t(np.concatenate([ctxs[b] for b in ids])), nxt_a)
    kvs, pending = [], []
    for b in range(B):
        kv = RequestKV(CFG)
        pending.append(prefill_request(CFG, W, kv, ctxs[b])["next"] if lens[b] else 7)
        kvs.append(kv)
    rng = np.random.default_rng(23)
    full = greedy_decode(CFG, W, copy.deepcopy(kvs[0]), pending[0], k)
    mixed = greedy_decode(CFG, W, copy.deepcopy(kvs[2]), pending[2], k)
    mixed[15] = (mixed[15] + 1) % CFG.vocab                   # the chain breaks at draft 16
    drafts = [full, [int(x) for x in rng.integers(0, CFG.vocab, k)], mixed]
    seq, ctx = _t(range(B)), _t(lens)
    acc, nxt = _t([0] * B), _t([0] * B)
    logits = torch.full((B * (k + 1), CFG.vocab), float("nan"), device=DEV)
    war.verify_step(model, pool, seq, ctx, _t(pending), _t(drafts), None, k, acc, nxt, logits)
    torch.cuda.synchronize()
    g_acc, g_nxt = acc.cpu().numpy(), nxt.cpu().numpy()
    glog = logits.cpu().numpy().reshape(B, k + 1, CFG.vocab)
    report = []
    for b in range(B):
        r = verify_request(CFG, W, kvs[b], pending[b], drafts[b])
        compare_request(r["logits"], glog[b], drafts[b], r["accept"], r["next"],
                        int(g_acc[b]), int(g_nxt[b]), report, f"request {b}")
    print(f"\naccept lengths {g_acc.tolist()}; reported: {report}")
    war.kv_commit(pool, seq, ctx, _t([-1] * B))
    # one more draft than the row block holds is refused before anything runs
    with pytest.raises(war.WarError):
        war.verify_step(model, pool, seq, ctx, _t(pending), _t(np.zeros((B, k + 1))), None, k + 1,
                        acc, nxt)
    torch.cuda.synchronize()
