"""Paged-KV bookkeeping model -- oracle (test infrastructure only).

The paper's rollout replicas keep each trajectory's KV cache and reuse it when
the next turn arrives; the footprint grows with the sequence and memory
pressure decides how much can stay resident (Background, "Rollout Bottlenecks";
System Design, "Overview of WAR").  The paper gives no layout or allocator.
The reading taken here, which the device allocator must reproduce bit for bit:

  * KV lives in fixed pages of ``page_size`` token slots; sequence s maps its
    logical page j to a physical page through block_table[s][j] (-1 = none);
  * free pages sit on a stack (top = end of the list), initialised so that
    pops return page ids 0, 1, 2, ...;
  * pops happen for batch entries in ascending order, logical pages ascending;
    pushes for batch entries in descending order, logical pages descending --
    so reserving and then discarding a step restores the stack exactly;
  * fork shares whole pages (n_tokens a multiple of page_size) and raises
    their reference counts; a page returns to the stack when its count hits 0;
  * a verify step reserves the pages needed for ctx + draft_len + 1 slots;
    commit with accept a keeps ctx + a + 1 tokens and returns the pages this
    step reserved beyond them (rollback); a = -1 discards the whole step.
Every operation validates first and changes nothing when it fails.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np


class PoolError(Exception):
    pass


def cdiv(a: int, b: int) -> int:
    return -(-a // b)


class PagePool:
    def __init__(self, num_pages: int, page_size: int, max_seqs: int, max_pages: int):
        self.P, self.num_pages = page_size, num_pages
        self.max_seqs, self.max_pages = max_seqs, max_pages
        self.stack: List[int] = list(range(num_pages - 1, -1, -1))
        self.refcount = np.zeros(num_pages, np.int32)
        self.table = np.full((max_seqs, max_pages), -1, np.int32)
        self.held = np.zeros(max_seqs, np.int32)
        self.base = np.zeros(max_seqs, np.int32)

    # ------------------------------------------------------------------ helpers
    @property
    def free_count(self) -> int:
        return len(self.stack)

    def _check_seqs(self, seq_ids: Sequence[int]) -> None:
        if len(set(int(s) for s in seq_ids)) != len(seq_ids):
            raise PoolError("duplicate sequence id")
        for s in seq_ids:
            if not 0 <= int(s) < self.max_seqs:
                raise PoolError(f"sequence id {s} out of range")

    def _grow(self, seq_ids, targets) -> None:
        """Pop pages so that seq_ids[b] holds targets[b] pages (b ascending)."""
        needs = [max(0, int(t) - int(self.held[s])) for s, t in zip(seq_ids, targets)]
        for t in targets:
            if int(t) > self.max_pages:
                raise PoolError("sequence exceeds max pages per sequence")
        if sum(needs) > self.free_count:
            raise PoolError("out of pages")
        for s, need in zip(seq_ids, needs):
            for _ in range(need):
                page = self.stack.pop()
                self.refcount[page] = 1
                self.table[s, self.held[s]] = page
                self.held[s] += 1

    def _shrink(self, s: int, keep: int) -> None:
        """Drop logical pages held-1 .. keep of sequence s (descending)."""
        for j in range(int(self.held[s]) - 1, keep - 1, -1):
            page = int(self.table[s, j])
            self.refcount[page] -= 1
            if self.refcount[page] == 0:
                self.stack.append(page)
            self.table[s, j] = -1
        self.held[s] = min(int(self.held[s]), keep)

    # --------------------------------------------------------------- operations
    def alloc(self, seq_ids: Sequence[int], n_tokens: Sequence[int]) -> None:
        """Ensure capacity for n_tokens slots per sequence."""
        self._check_seqs(seq_ids)
        if any(int(n) < 0 for n in n_tokens):
            raise PoolError("negative token count")
        self._grow(seq_ids, [cdiv(int(n), self.P) for n in n_tokens])
        for s in seq_ids:
            self.base[s] = self.held[s]

    def fork(self, src: int, dst: int, n_tokens: int) -> None:
        """dst shares the first n_tokens (whole pages) of src."""
        self._check_seqs([src, dst])
        if n_tokens % self.P or n_tokens < 0:
            raise PoolError("fork length must be a multiple of the page size")
        npg = n_tokens // self.P
        if self.held[dst] != 0 or self.held[src] < npg:
            raise PoolError("bad fork")
        for j in range(npg):
            page = int(self.table[src, j])
            self.table[dst, j] = page
            self.refcount[page] += 1
        self.held[dst] = npg
        self.base[dst] = npg

    def free(self, seq_ids: Sequence[int]) -> None:
        self._check_seqs(seq_ids)
        for s in reversed(list(seq_ids)):
            self._shrink(int(s), 0)
            self.base[s] = 0

    def reserve(self, seq_ids, ctx_lens, draft_lens) -> None:
        """Verify step: room for ctx + draft_len + 1 slots per entry."""
        self._check_seqs(seq_ids)
        targets = [cdiv(int(c) + int(n) + 1, self.P) for c, n in zip(ctx_lens, draft_lens)]
        self._grow_step(seq_ids, targets)

    def _grow_step(self, seq_ids, targets) -> None:
        before = [int(self.held[s]) for s in seq_ids]
        self._grow(seq_ids, targets)
        for s, h in zip(seq_ids, before):
            self.base[s] = h

    def commit(self, seq_ids, ctx_lens, accept_lens) -> np.ndarray:
        """Keep ctx + a + 1 tokens (a = -1: keep ctx); return the new ctx_lens."""
        self._check_seqs(seq_ids)
        ctx = np.array(ctx_lens, dtype=np.int64)
        for b in range(len(seq_ids) - 1, -1, -1):
            s = int(seq_ids[b])
            cap = int(self.held[s]) * self.P
            a = max(-1, min(int(accept_lens[b]), cap - int(ctx[b]) - 1))
            new_ctx = int(ctx[b]) + a + 1
            keep = min(int(self.held[s]), max(int(self.base[s]), cdiv(new_ctx, self.P)))
            self._shrink(s, keep)
            self.base[s] = self.held[s]
            ctx[b] = new_ctx
        return ctx.astype(np.int32)

    def prefill_reserve(self, seq_ids, ctx_lens, n_new) -> None:
        """Append: room for ctx + n_new slots per entry."""
        self._check_seqs(seq_ids)
        self._grow(seq_ids, [cdiv(int(c) + int(n), self.P) for c, n in zip(ctx_lens, n_new)])
        for s in seq_ids:
            self.base[s] = self.held[s]

    # ----------------------------------------------------------------- queries
    def snapshot(self) -> Dict[str, np.ndarray]:
        return {"stack": np.array(self.stack, dtype=np.int32),
                "refcount": self.refcount.copy(), "table": self.table.copy(),
                "held": self.held.copy(), "base": self.base.copy()}

    def slot(self, s: int, pos: int) -> tuple:
        """(physical page, offset) of token position pos of sequence s."""
        return int(self.table[s, pos // self.P]), pos % self.P

    def check_invariants(self) -> None:
        """Every page is either free (exactly once) or referenced by block tables
        exactly refcount times; block tables hold pages only below ``held``."""
        counts = np.zeros(self.num_pages, np.int64)
        for s in range(self.max_seqs):
            h = int(self.held[s])
            row = self.table[s]
            assert (row[h:] == -1).all(), "entry beyond held"
            assert (row[:h] >= 0).all(), "hole below held"
            np.add.at(counts, row[:h], 1)
        assert (counts == self.refcount).all(), "refcount mismatch"
        free = np.zeros(self.num_pages, np.int64)
        np.add.at(free, np.array(self.stack, dtype=np.int64), 1)
        assert (free <= 1).all(), "page on the stack twice"
        assert ((free == 1) == (counts == 0)).all(), "page both free and used (or lost)"
