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
