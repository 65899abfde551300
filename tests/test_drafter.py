"""The host suffix-match drafter against a brute-force scan, and on motif data."""
import numpy as np

from paper_2607_17299_amd import synth
from paper_2607_17299_amd.drafter import SuffixDrafter, brute_force_propose


def test_drafter_matches_brute_force_on_tiny_corpora():
    rng = np.random.default_rng(0)
    for trial in range(300):
        vocab = int(rng.integers(2, 5))
        trajs = [rng.integers(0, vocab, int(rng.integers(0, 25))).tolist()
                 for _ in range(int(rng.integers(1, 4)))]
        ctx = rng.integers(0, vocab, int(rng.integers(0, 12))).tolist()
        k = int(rng.integers(0, 6))
        mm = int(rng.integers(1, 8))
        d = SuffixDrafter(max_match=mm)
        for t in trajs:
            d.add_trajectory(t)
        assert d.propose(ctx, k) == brute_force_propose(trajs, ctx, k, mm), trial


def test_drafter_continues_a_motif():
    bank = synth.MotifBank(seed=1, vocab=4096, n_motifs=16)
    d = SuffixDrafter()
    for i in range(8):
        d.add_trajectory(bank.trajectory(100 + i, 4096))
    m = bank.motifs[3]
    d.add_trajectory(m)
    ctx = np.concatenate([synth.uniform_tokens(3, 50, 4096), m[:40]])
    assert d.propose(ctx, 8) == m[40:48].tolist()


def test_drafter_no_match_gives_no_draft():
    d = SuffixDrafter()
    d.add_trajectory([1, 2, 3])
    assert d.propose([7, 8], 4) == []
    assert d.propose([3], 4) == []          # 3 ends its trajectory: nothing follows
    assert d.propose([1], 4) == [2, 3]


def test_tree_drafter_matches_brute_force_on_tiny_corpora():
    from paper_2607_17299_amd.drafter import brute_force_propose_tree
    rng = np.random.default_rng(1)
    for trial in range(200):
        vocab = int(rng.integers(2, 5))
        trajs = [rng.integers(0, vocab, int(rng.integers(0, 25))).tolist()
                 for _ in range(int(rng.integers(1, 4)))]
        ctx = rng.integers(0, vocab, int(rng.integers(0, 12))).tolist()
        n = int(rng.integers(0, 8))
        mm = int(rng.integers(1, 8))
        d = SuffixDrafter(max_match=mm)
        for t in trajs:
            d.add_trajectory(t)
        toks, par = d.propose_tree(ctx, n)
        assert (toks, par) == brute_force_propose_tree(trajs, ctx, n, mm), trial
        assert len(toks) <= n and all(0 <= p <= i for i, p in enumerate(par))
        # the first node is the chain drafter's first token
        assert toks[:1] == d.propose(ctx, min(n, 1))


def test_tree_drafter_on_a_unique_continuation_is_the_chain():
    d = SuffixDrafter()
    d.add_trajectory(list(range(100, 140)))
    toks, par = d.propose_tree([5, 100, 101], 6)
    assert toks == d.propose([5, 100, 101], 6) == list(range(102, 108))
    assert par == list(range(6))


def test_tree_drafter_branches_on_diverging_histories():
    d = SuffixDrafter()
    for _ in range(3):
        d.add_trajectory([1, 2, 3, 4, 5])
    d.add_trajectory([1, 2, 7, 8])
    toks, par = d.propose_tree([9, 1, 2], 4)
    # 3 (share 3/4) then its child 4 (3/4) then 7 (1/4, proposed before 5) ...
    assert toks[:2] == [3, 4] and par[:2] == [0, 1]
    assert (7, 0) in list(zip(toks, par))
