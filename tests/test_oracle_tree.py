"""Pins of the oracle's tree-draft verification (CPU, tiny decoder)."""
import numpy as np
import pytest

from oracle.accept import argmax_lowest
from oracle.decoder import RequestKV, Weights
from oracle.verify import (commit_request, greedy_decode, prefill_request, tree_path, verify_request,
                           verify_tree_request)
from paper_2607_17299_amd import synth

CFG = synth.TINY


@pytest.fixture(scope="module")
def env():
    W = Weights(CFG, synth.model_weights(CFG, seed=0, norm_std=0.1))
    kv = RequestKV(CFG)
    r = prefill_request(CFG, W, kv, synth.uniform_tokens(31, 96, CFG.vocab))
    return W, kv, r["next"]


def _copy(kv):
    return RequestKV(CFG, list(kv.layers))


def test_chain_tree_equals_chain_verify(env):
    W, kv, x = env
    drafts = [int(t) for t in synth.uniform_tokens(32, 5, CFG.vocab)]
    rc = verify_request(CFG, W, _copy(kv), x, drafts)
    rt = verify_tree_request(CFG, W, _copy(kv), x, drafts, [0, 1, 2, 3, 4])
    np.testing.assert_allclose(rt["logits"], rc["logits"], atol=1e-9)
    assert (rt["accept"], rt["next"]) == (rc["accept"], rc["next"])
    assert rt["path"] == list(range(1, rc["accept"] + 1))


def test_node_logits_equal_the_chain_verify_of_their_path(env):
    W, kv, x = env
    rng = np.random.default_rng(3)
    n = 7
    parents = [int(rng.integers(0, j + 1)) for j in range(n)]
    drafts = [int(t) for t in rng.integers(0, CFG.vocab, n)]
    rt = verify_tree_request(CFG, W, _copy(kv), x, drafts, parents)
    for j in range(1, n + 1):
        p = tree_path(parents, j)
        rc = verify_request(CFG, W, _copy(kv), x, [drafts[i - 1] for i in p[1:]])
        np.testing.assert_allclose(rt["logits"][j], rc["logits"][-1], atol=1e-9)


def test_greedy_branch_is_accepted_among_distractors(env):
    """A tree whose branches include the greedy continuation accepts exactly it
    (losslessness: the emitted tokens are token-by-token greedy decode)."""
    W, kv, x = env
    g = greedy_decode(CFG, W, _copy(kv), x, 4)           # tokens after x
    rng = np.random.default_rng(4)
    other = [int(t) for t in rng.integers(0, CFG.vocab, 3)]
    # node 1: a distractor; node 2: g[0]; node 3: child of 1; node 4: g[1] under 2;
    # node 5: a distractor under 2; node 6: g[2] under 4
    drafts = [other[0], g[0], other[1], g[1], other[2], g[2]]
    parents = [0, 0, 1, 2, 2, 4]
    r = verify_tree_request(CFG, W, _copy(kv), x, drafts, parents)
    assert r["path"] == [2, 4, 6] and r["accept"] == 3 and r["next"] == g[3]
    kv2 = _copy(kv)
    commit_request(kv2, r)
    assert kv2.length == kv.length + 4
    rc = verify_request(CFG, W, _copy(kv), x, g[:3])
    for l in range(CFG.n_layers):
        np.testing.assert_allclose(r["new_kv"][l][0], rc["new_kv"][l][0], atol=1e-9)


def _brute_path(parents, tok, g):
    """Enumerate every root-to-node path; keep the longest whose every node
    carries its parent's greedy token, ties broken by the lowest end node."""
    best = []
    for j in range(len(tok)):
        p = tree_path(parents, j)[1:]
        ok = all(tok[c] == g[([0] + p)[k]] for k, c in enumerate(p))
        if ok and len(p) > len(best):
            best = p
    return best


def test_acceptance_against_path_enumeration(env):
    W, kv, x = env
    base = verify_request(CFG, W, _copy(kv), x, [])
    g0 = int(base["greedy"][0])
    rng = np.random.default_rng(5)
    for trial in range(6):
        n = 6
        parents = [int(rng.integers(0, j + 1)) for j in range(n)]
        # bias tokens towards the greedy choice so that paths get accepted
        drafts = [g0 if (parents[j] == 0 and rng.random() < 0.7) else int(rng.integers(CFG.vocab))
                  for j in range(n)]
        r = verify_tree_request(CFG, W, _copy(kv), x, drafts, parents)
        g = argmax_lowest(r["logits"])
        assert r["path"] == _brute_path(parents, [x] + drafts, g), (trial, parents, drafts)
        assert r["accept"] == len(r["path"]) and r["next"] == int(g[([0] + r["path"])[-1]])


def test_duplicate_siblings_take_the_deeper_branch(env):
    """Two siblings carry the same (greedy) token; only the second has the
    greedy continuation below it, so the deeper path goes through it."""
    W, kv, x = env
    g = greedy_decode(CFG, W, _copy(kv), x, 3)
    wrong = (g[1] + 1) % CFG.vocab
    drafts = [g[0], g[0], wrong, g[1]]
    parents = [0, 0, 1, 2]
    r = verify_tree_request(CFG, W, _copy(kv), x, drafts, parents)
    assert r["path"] == [2, 4] and r["next"] == g[2]
    # equal depths: the lowest end node wins
    r = verify_tree_request(CFG, W, _copy(kv), x, [g[0], g[0]], [0, 0])
    assert r["path"] == [1]
