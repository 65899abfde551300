"""GPU checks of the boundary's failure handling on the tiny decoder.

* A verify step whose device-side inputs are bad (a sequence id repeated in
  the batch, or one request past its block-table row) fails as a whole: no
  page moves, every accept length and next token is -1, the following commit
  changes nothing whatever accept lengths it is given, and war_pool_state
  reports WAR_ERR_DEVICE once, then clears the flag.
* A steady verify/commit loop never waits for the device to learn how many
  pages are free: the commit kernel's report keeps the host's lower bound up.
All failure conditions are plain inputs that the kernels' own checks turn
into flags; every kernel runs to completion.
"""
import numpy as np
import pytest
import torch

from paper_2607_17299_amd import synth

pytestmark = pytest.mark.gpu
CFG = synth.TINY
DEV = "cuda"


def _war():
    from paper_2607_17299_amd import war
    return war


@pytest.fixture(scope="module")
def tiny():
    war = _war()
    w = {k: v.to(DEV) for k, v in synth.model_weights(CFG, seed=0, norm_std=0.1).items()}
    return war, war.Model(CFG, w, max_rows=64)


def _t(a):
    return torch.as_tensor(np.asarray(a), dtype=torch.int32).to(DEV)


def _prefilled(war, model, lens, num_pages=64, max_pages=8):
    B = len(lens)
    pool = war.Pool(CFG, num_pages, B + 1, max_pages)
    ctx = _t([0] * B)
    toks = _t(np.concatenate([synth.uniform_tokens(300 + b, n, CFG.vocab) for b, n in enumerate(lens)]))
    nxt = _t([0] * B)
    war.prefill_append(model, pool, _t(range(B)), ctx, list(lens), toks, nxt)
    torch.cuda.synchronize()
    return pool, ctx, nxt


def _snapshot(pool):
    st = pool.state()
    assert st["status"] == 0
    return {k: st[k].copy() for k in ("stack", "refcount", "held", "base", "table")}


def _flagged(war, pool, words):
    """war_pool_state reports the device's flag once (WAR_ERR_DEVICE)."""
    st = pool.state()
    assert st["status"] == -5
    assert words in war.lib().war_last_error().decode()


def _same(a, b):
    for k in a:
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def _failed_step(war, model, pool, seq, ctx, last, k, commit_with):
    B = seq.numel()
    drafts = _t(np.arange(B * k).reshape(B, k) % CFG.vocab)
    acc, nxt = _t([7] * B), _t([7] * B)
    ctx_before = ctx.cpu().tolist()
    war.verify_step(model, pool, seq, ctx, last, drafts, None, k, acc, nxt)
    war.kv_commit(pool, seq, ctx, acc if commit_with is None else _t(commit_with))
    torch.cuda.synchronize()
    assert acc.cpu().tolist() == [-1] * B
    assert nxt.cpu().tolist() == [-1] * B
    assert ctx.cpu().tolist() == ctx_before


@pytest.mark.parametrize("commit_with", [None, [3, 3, 3]])
def test_repeated_sequence_id_fails_the_step(tiny, commit_with):
    war, model = tiny
    pool, ctx, nxt = _prefilled(war, model, [40, 37, 50])
    before = _snapshot(pool)
    seq = _t([0, 1, 0])
    _failed_step(war, model, pool, seq, ctx, nxt, 4, commit_with)
    _flagged(war, pool, "twice")
    _same(before, _snapshot(pool))                     # flag cleared, nothing moved
    # the pool still works: a valid step on the same sequences
    acc, nx = _t([0] * 3), _t([0] * 3)
    seq = _t([0, 1, 2])
    war.verify_step(model, pool, seq, ctx, nxt, _t([[1, 2]] * 3), None, 2, acc, nx)
    war.kv_commit(pool, seq, ctx, _t([-1] * 3))
    torch.cuda.synchronize()
    assert min(acc.cpu().tolist()) >= 0
    _same(before, _snapshot(pool))


@pytest.mark.parametrize("commit_with", [None, [4, 4, 4]])
def test_request_past_its_block_table_fails_the_step(tiny, commit_with):
    """max_pages_per_seq = 4 (64 slots): request 1 has 60 cached tokens, so
    60 + 4 drafts + 1 > 64 fails the whole batch."""
    war, model = tiny
    pool, ctx, nxt = _prefilled(war, model, [20, 60, 33], max_pages=4)
    before = _snapshot(pool)
    _failed_step(war, model, pool, _t([0, 1, 2]), ctx, nxt, 4, commit_with)
    _flagged(war, pool, "context length")
    _same(before, _snapshot(pool))


def test_bad_sequence_id_fails_the_step(tiny):
    war, model = tiny
    pool, ctx, nxt = _prefilled(war, model, [20, 30])
    before = _snapshot(pool)
    _failed_step(war, model, pool, _t([0, 99]), ctx, nxt, 2, [1, 1])
    _flagged(war, pool, "sequence id")
    _same(before, _snapshot(pool))


def test_steady_loop_never_waits_for_the_free_count(tiny):
    """4 requests x k = 4 reserve at most 4 pages per step; the pool has 40
    free pages, so a bound that only fell would need an exact read within 10
    steps.  Over 60 steps (each followed by a host synchronisation, so that
    the commit report is current) no verify step reads the exact count."""
    war, model = tiny
    pool, ctx, nxt = _prefilled(war, model, [20, 30, 16, 45], num_pages=48)
    seq = _t(range(4))
    acc, nx = _t([0] * 4), _t([0] * 4)
    drafts = _t(np.arange(16).reshape(4, 4))
    free0 = pool.state()["stack"].size
    assert free0 == 48 - (2 + 2 + 1 + 3)
    w0 = pool.waits()
    for _ in range(60):
        war.verify_step(model, pool, seq, ctx, nxt, drafts, None, 4, acc, nx)
        war.kv_commit(pool, seq, ctx, _t([-1] * 4))
        torch.cuda.synchronize()
    assert pool.waits() == w0
    assert pool.state()["stack"].size == free0
