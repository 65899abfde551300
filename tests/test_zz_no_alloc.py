"""war_verify_step_noalloc, the verify step laid over the library's static
device scratch, against war_verify_step through the C ABI: the same accept
lengths, next tokens, logits and written KV, bit for bit (the same kernels,
splits and attention chunks over the same inputs), on two calls in a row, the
second with a smaller batch.  A step whose workspace exceeds the scratch is
refused before anything is enqueued."""
import numpy as np
import pytest
import torch

from paper_2607_17299_amd import harness, synth

pytestmark = pytest.mark.gpu
KV_SEED = 9


def _war():
    from paper_2607_17299_amd import war
    return war


def _once(war, fn, model, pool, cfg, st):
    """One call of fn (either entry point), its outputs and the KV it wrote
    (read back before the discarding commit)."""
    ds = harness.DeviceStep(st, with_logits=True, vocab=cfg.vocab)
    ds.logits.fill_(float("nan"))
    fn(model, pool, ds.seq, ds.ctx, ds.last, ds.drafts, ds.dlens, st.k_max, ds.accept, ds.next, ds.logits)
    torch.cuda.synchronize()
    kv = [pool.gather_kv(int(s), int(c) + len(d) + 1, l)[:, :, int(c):].clone()
          for s, c, d in zip(st.seq_ids, st.ctx_lens, st.drafts) for l in range(cfg.n_layers)]
    out = {"accept": ds.accept.cpu().clone(), "next": ds.next.cpu().clone(), "kv": kv}
    rows = [b * (st.k_max + 1) + i for b, d in enumerate(st.drafts) for i in range(len(d) + 1)]
    out["logits"] = ds.logits[rows].cpu().clone()
    ds.commit(pool, discard=True)
    torch.cuda.synchronize()
    return out


def _same(a, b):
    assert torch.equal(a["accept"], b["accept"]) and torch.equal(a["next"], b["next"])
    assert torch.equal(a["logits"].view(torch.int32), b["logits"].view(torch.int32))
    for x, y in zip(a["kv"], b["kv"]):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))


def _step(seed, B, k, ctxs, vocab):
    rng = np.random.default_rng(seed)
    drafts = [rng.integers(0, vocab, int(rng.integers(0, k + 1))).tolist() for _ in range(B)]
    return harness.Step(np.arange(B, dtype=np.int32), np.asarray(ctxs[:B], np.int32),
                        synth.uniform_tokens(seed + 1, B, vocab), drafts, k)


def test_noalloc_matches_verify_step_at_full_widths():
    """2 layers of the 36-layer shapes: 8 requests with k = 8 (72 rows, three
    query-row tiles) over 1500-4500 cached tokens, then 3 requests with k = 2."""
    war = _war()
    cfg = synth.reduced(synth.LARGE, 2)
    model = war.Model(cfg, harness.large_weights(cfg), max_rows=512)
    ctxs = np.array([4500, 1500, 3001, 2048, 2700, 4097, 1999, 3333], np.int32)
    pool = harness.make_pool(cfg, ctxs, 10)
    harness.load_contexts(pool, cfg, ctxs, np.arange(8), KV_SEED)
    before = pool.state()
    for st in (_step(3, 8, 8, ctxs, cfg.vocab), _step(4, 3, 2, ctxs, cfg.vocab)):
        print(f"noalloc vs verify_step: B={st.B} k={st.k_max}", flush=True)
        ref = _once(war, war.verify_step, model, pool, cfg, st)
        got = _once(war, war.verify_step_noalloc, model, pool, cfg, st)
        _same(ref, got)
    after = pool.state()
    for key in ("stack", "refcount", "held", "base", "table"):
        np.testing.assert_array_equal(before[key], after[key])


def test_noalloc_matches_verify_step_on_the_tiny_decoder():
    war = _war()
    cfg = synth.TINY
    w = {k: v.cuda() for k, v in synth.model_weights(cfg, seed=0, norm_std=0.1).items()}
    model = war.Model(cfg, w, max_rows=64)
    ctxs = np.array([300, 77, 512, 129], np.int32)
    pool = harness.make_pool(cfg, ctxs, 6)
    harness.load_contexts(pool, cfg, ctxs, np.arange(4), KV_SEED)
    for st in (_step(5, 4, 5, ctxs, cfg.vocab), _step(6, 2, 1, ctxs, cfg.vocab)):
        print(f"noalloc vs verify_step (tiny): B={st.B} k={st.k_max}", flush=True)
        _same(_once(war, war.verify_step, model, pool, cfg, st),
              _once(war, war.verify_step_noalloc, model, pool, cfg, st))


def test_noalloc_refuses_a_step_beyond_the_scratch():
    """64 requests x k = 11 (768 rows) at full widths need about 90 MB of
    workspace, more than the 64 MiB scratch: refused with
    WAR_ERR_UNSUPPORTED, nothing enqueued."""
    war = _war()
    cfg = synth.reduced(synth.LARGE, 1)
    model = war.Model(cfg, harness.large_weights(cfg), max_rows=1024)
    B = 64
    pool = war.Pool(cfg, 256, B, 8)
    before = pool.state()
    t = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.int32).cuda()
    acc, nxt = t([0] * B), t([0] * B)
    with pytest.raises(war.WarError) as e:
        war.verify_step_noalloc(model, pool, t(range(B)), t([0] * B), t([1] * B), t(np.ones((B, 11))),
                                None, 11, acc, nxt)
    assert e.value.status == -4 and "scratch" in str(e.value)
    after = pool.state()
    for key in ("stack", "refcount", "held", "base", "table"):
        np.testing.assert_array_equal(before[key], after[key])
