"""Speculation on/off policy (host logic, no GPU)."""
import itertools

import pytest

from oracle.accept import accept_length
from paper_2607_17299_amd.policy import SpecPolicy, expected_tokens


@pytest.mark.parametrize("k", [0, 1, 2, 4, 8])
@pytest.mark.parametrize("alpha", [0.0, 0.3, 0.8, 1.0])
def test_expected_tokens_matches_enumeration_of_the_prefix_rule(k, alpha):
    """Enumerate every pattern of per-draft matches, apply the oracle's
    acceptance rule to it, and weight by its probability."""
    total = 0.0
    for pat in itertools.product([True, False], repeat=k):
        p = 1.0
        for hit in pat:
            p *= alpha if hit else 1 - alpha
        drafts = list(range(k))
        greedy = [d if hit else -1 for d, hit in zip(drafts, pat)] + [-1]
        total += p * (accept_length(drafts, greedy) + 1)
    assert expected_tokens(k, alpha) == pytest.approx(total, rel=1e-12, abs=1e-12)


def test_expected_tokens_special_cases():
    assert expected_tokens(0, 0.7) == 1.0
    assert expected_tokens(5, 1.0) == 6.0
    assert expected_tokens(5, 0.0) == 1.0
    with pytest.raises(ValueError):
        expected_tokens(-1, 0.5)


def _table():
    # step time = launch-bound floor + per-row cost: speculation is cheap at
    # small batches and costly at large ones
    t = {}
    for b in [1, 2, 4, 8, 16, 32, 64]:
        for k in [0, 2, 4, 8]:
            t[(b, k)] = 10.0 + 0.5 * b * (k + 1)
    return t


def test_choose_k_switches_off_at_large_batches():
    pol = SpecPolicy(_table())
    assert pol.choose_k(1, 0.8) > 0
    assert pol.choose_k(64, 0.8) == 0
    assert pol.choose_k(64, 0.0) == 0           # nothing accepted: never speculate
    c = pol.crossover(0.8)
    assert c is not None and 1 <= c < 64
    # a better acceptance rate keeps speculation on up to larger batches
    assert pol.crossover(0.95) >= c


def test_interpolation_and_validation():
    pol = SpecPolicy(_table())
    assert pol.time_ms(1, 0) == 10.5
    assert pol.time_ms(100, 0) == pol.time_ms(64, 0)
    mid = pol.time_ms(6, 2)
    assert pol.time_ms(4, 2) < mid < pol.time_ms(8, 2)
    bad = _table()
    del bad[(8, 4)]
    with pytest.raises(ValueError):
        SpecPolicy(bad)
