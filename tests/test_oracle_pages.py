"""Pins of the paged-KV bookkeeping model: hand-worked cases, invariants under
random operation sequences, exact restoration by discard, and brute-force
enumeration of every short operation sequence on a tiny pool."""
import itertools

import numpy as np
import pytest

from oracle.pages import PagePool, PoolError, cdiv


def test_hand_worked_sequence():
    p = PagePool(num_pages=8, page_size=16, max_seqs=3, max_pages=5)
    p.alloc([0, 1], [40, 20])            # seq0: 3 pages, seq1: 2 pages
    assert p.table[0, :3].tolist() == [0, 1, 2] and p.table[1, :2].tolist() == [3, 4]
    p.fork(0, 2, 32)                     # seq2 shares pages 0, 1
    assert p.table[2, :2].tolist() == [0, 1] and p.refcount[:3].tolist() == [2, 2, 1]
    p.free([0])                          # page 2 back; 0, 1 still used by seq2
    assert p.stack[-1] == 2 and p.refcount[:3].tolist() == [1, 1, 0]
    # verify reserve: seq2 ctx 32 + 3 drafts + 1 -> 3 pages (1 new); seq1 ctx 20 + 0 + 1 -> 2 pages
    p.reserve([2, 1], [32, 20], [3, 0])
    assert p.table[2, :3].tolist() == [0, 1, 2]
    # accept 1 -> ctx 34 keeps 3 pages; seq1 accept 0 -> ctx 21 keeps 2
    ctx = p.commit([2, 1], [32, 20], [1, 0])
    assert ctx.tolist() == [34, 21] and p.held[2] == 3
    p.check_invariants()


def test_discard_restores_state_exactly():
    rng = np.random.default_rng(0)
    p = PagePool(num_pages=64, page_size=4, max_seqs=6, max_pages=16)
    p.alloc(list(range(6)), rng.integers(1, 30, 6).tolist())
    ctx = [int(cdiv(int(h) * 4, 1)) - int(rng.integers(0, 4)) for h in p.held]
    before = p.snapshot()
    p.reserve(list(range(6)), ctx, rng.integers(0, 9, 6).tolist())
    p.commit(list(range(6)), ctx, [-1] * 6)
    after = p.snapshot()
    for k in before:
        if k != "base":
            np.testing.assert_array_equal(before[k], after[k])


def test_rollback_returns_only_step_pages():
    p = PagePool(num_pages=32, page_size=4, max_seqs=2, max_pages=16)
    p.alloc([0], [20])                   # capacity for 20 tokens (5 pages), ctx is 9
    p.reserve([0], [9], [8])             # needs 18 slots -> 5 pages: nothing new
    assert p.held[0] == 5
    p.commit([0], [9], [0])              # keeps ctx 10: the alloc'd pages stay
    assert p.held[0] == 5
    p.reserve([0], [10], [12])           # 23 slots -> 6 pages, one new
    ctx = p.commit([0], [10], [2])       # ctx 13 -> 4 pages needed, but alloc'd 5 stay
    assert ctx[0] == 13 and p.held[0] == 5
    p.check_invariants()


def test_errors_change_nothing():
    p = PagePool(num_pages=4, page_size=4, max_seqs=3, max_pages=3)
    p.alloc([0], [8])
    s = p.snapshot()
    for bad in (lambda: p.alloc([1], [40]),           # more than max pages
                lambda: p.alloc([1, 2], [12, 12]),    # out of pages
                lambda: p.alloc([1, 1], [4, 4]),      # duplicate id
                lambda: p.fork(0, 1, 6),              # not page aligned
                lambda: p.fork(0, 0, 4),              # dst not empty
                lambda: p.reserve([0, 1], [8, 0], [4, 8]),
                lambda: p.alloc([5], [4])):
        with pytest.raises(PoolError):
            bad()
        t = p.snapshot()
        for k in s:
            np.testing.assert_array_equal(s[k], t[k])


def _random_ops(p, rng, n_ops, ctx):
    S = p.max_seqs
    for _ in range(n_ops):
        op = rng.integers(0, 5)
        ids = rng.permutation(S)[: int(rng.integers(1, S + 1))].tolist()
        try:
            if op == 0:
                n = rng.integers(0, p.max_pages * p.P, len(ids)).tolist()
                p.alloc(ids, n)
                for s, t in zip(ids, n):
                    ctx[s] = min(max(ctx[s], 0), int(p.held[s]) * p.P)
            elif op == 1:
                src, dst = int(rng.integers(S)), int(rng.integers(S))
                n = int(rng.integers(0, p.held[src] + 1)) * p.P
                p.fork(src, dst, n)
                ctx[dst] = n
            elif op == 2:
                p.free(ids)
                for s in ids:
                    ctx[s] = 0
            else:
                d = rng.integers(0, 5, len(ids)).tolist()
                c = [ctx[s] for s in ids]
                p.reserve(ids, c, d)
                acc = [int(rng.integers(-1, di + 1)) for di in d]
                new = p.commit(ids, c, acc)
                for s, v in zip(ids, new):
                    ctx[s] = int(v)
        except PoolError:
            pass
        p.check_invariants()


def test_invariants_under_random_operation_sequences():
    for seed in range(40):
        rng = np.random.default_rng(seed)
        p = PagePool(num_pages=int(rng.integers(4, 40)), page_size=int(rng.choice([1, 2, 4, 16])),
                     max_seqs=int(rng.integers(1, 6)), max_pages=int(rng.integers(1, 12)))
        _random_ops(p, rng, 60, [0] * p.max_seqs)


def test_brute_force_all_short_sequences_on_tiny_pool():
    # Every sequence of 3 operations from a small alphabet, 3 pages, 2 sequences.
    alphabet = []
    for s in (0, 1):
        for n in (0, 1, 3):
            alphabet.append(("alloc", s, n))
        alphabet.append(("free", s, 0))
        for d in (0, 1, 2):
            for a in (-1, 0, 1):
                alphabet.append(("step", s, (d, a)))
    alphabet.append(("fork", 0, 1))
    alphabet.append(("fork", 1, 0))
    count = 0
    for seq in itertools.product(alphabet, repeat=3):
        p = PagePool(num_pages=3, page_size=1, max_seqs=2, max_pages=3)
        ctx = [0, 0]
        for op, s, arg in seq:
            try:
                if op == "alloc":
                    p.alloc([s], [arg])
                elif op == "free":
                    p.free([s]); ctx[s] = 0
                elif op == "fork":
                    p.fork(s, arg, int(p.held[s])); ctx[arg] = int(p.held[s])
                else:
                    d, a = arg
                    c = min(ctx[s], int(p.held[s]))
                    p.reserve([s], [c], [d])
                    ctx[s] = int(p.commit([s], [c], [min(a, d)])[0])
                    assert ctx[s] == c + min(a, d) + 1
                    assert p.held[s] >= cdiv(ctx[s], 1)
            except PoolError:
                pass
            p.check_invariants()
            count += 1
    assert count == len(alphabet) ** 3 * 3
