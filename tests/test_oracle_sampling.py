"""Pins of the sampled-verification oracle (CPU)."""
import numpy as np
import pytest
import torch

from oracle.accept import accept_length, argmax_lowest
from oracle.sampling import filtered_probs, inverse_cdf, kept_tokens, verify_sampled


def test_kept_tokens_against_torch_topk_and_ties():
    rng = np.random.default_rng(0)
    z = rng.standard_normal(1000)
    keep = kept_tokens(z, 200)
    ref = torch.topk(torch.from_numpy(z), 200).indices.numpy()
    assert sorted(keep.tolist()) == sorted(ref.tolist())
    # ties at the boundary go to the lowest ids
    z = np.array([1.0, 3.0, 2.0, 2.0, 2.0, 0.5])
    assert kept_tokens(z, 3).tolist() == [1, 2, 3]
    assert kept_tokens(z, 10).tolist() == list(range(6))


@pytest.mark.parametrize("T", [1.0, 0.7, 1.5])
def test_filtered_probs_against_torch(T):
    rng = np.random.default_rng(1)
    z = rng.standard_normal(5000) * 3
    p = filtered_probs(z, T, 200)
    zt = torch.from_numpy(z)
    v, i = torch.topk(zt, 200)
    ref = torch.zeros_like(zt)
    ref[i] = torch.softmax(v / T, dim=0)
    np.testing.assert_allclose(p, ref.numpy(), rtol=1e-12, atol=1e-15)
    assert p.sum() == pytest.approx(1.0, abs=1e-12)


def test_inverse_cdf_against_brute_force():
    rng = np.random.default_rng(2)
    for _ in range(200):
        w = rng.random(17) * (rng.random(17) < 0.6)
        if w.sum() == 0:
            continue
        v = rng.random()
        acc, want = 0.0, None
        for t, x in enumerate(w):
            acc += x
            if acc > v * w.sum():
                want = t
                break
        assert inverse_cdf(w, v) == want


def test_top_k_one_is_greedy():
    """With one kept token the target is a point mass on the argmax: drafts are
    accepted exactly while they match it, whatever the uniforms."""
    rng = np.random.default_rng(3)
    for _ in range(100):
        n = int(rng.integers(0, 6))
        logits = rng.standard_normal((n + 1, 50))
        g = argmax_lowest(logits)
        drafts = [int(g[i]) if rng.random() < 0.6 else int(rng.integers(50)) for i in range(n)]
        r = verify_sampled(logits, drafts, rng.random(n + 1), rng.random(n + 1), 1.0, 1)
        a = accept_length(drafts, g)
        assert (r["accept"], r["next"]) == (a, int(g[a]))


def test_low_temperature_is_greedy():
    rng = np.random.default_rng(4)
    for _ in range(50):
        logits = rng.standard_normal((4, 30))
        g = argmax_lowest(logits)
        drafts = [int(g[0]), int(g[1]), int(rng.integers(30))]
        r = verify_sampled(logits, drafts, rng.random(4), rng.random(4), 1e-4, 200)
        a = accept_length(drafts, g)
        assert (r["accept"], r["next"]) == (a, int(g[a]))


def test_lossless_against_sequential_sampling():
    """Losslessness: a toy target whose next-token distribution depends on the
    previous token (a fixed 6 x 6 logit table).  Over many draws of the
    uniforms, the j-th emitted token, among runs whose first j-1 emitted tokens
    are the drafts d_1..d_{j-1}, must follow the target's conditional
    distribution after d_{j-1}.  A wrong acceptance test or a residual that
    does not remove the rejected draft shifts these frequencies by far more
    than the sampling error."""
    rng = np.random.default_rng(5)
    V, T, top_k = 6, 1.0, 4
    table = rng.standard_normal((V, V)) * 2.5
    x, drafts = 0, []
    for _ in range(3):          # the target's most likely chain: often, not always, accepted
        drafts.append(int(np.argmax(table[drafts[-1] if drafts else x])))
    rows = [table[x]] + [table[d] for d in drafts]
    logits = np.stack(rows)
    probs = [filtered_probs(r, T, top_k) for r in rows]
    N = 60000
    emitted = []
    for _ in range(N):
        r = verify_sampled(logits, drafts, rng.random(4), rng.random(4), T, top_k)
        emitted.append(drafts[: r["accept"]] + [r["next"]])
    for j in range(4):          # position j+1, conditioned on the prefix d_1..d_j
        sel = [e[j] for e in emitted if len(e) > j and e[:j] == drafts[:j]]
        n = len(sel)
        assert n > 500
        emp = np.bincount(sel, minlength=V) / n
        p = probs[j]
        tol = 5 * np.sqrt(p * (1 - p) / n) + 1e-9
        assert np.all(np.abs(emp - p) <= tol), (j, emp, p)
