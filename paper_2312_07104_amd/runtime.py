"""Host side of the hot path: Algorithm 1's per-request steps on the native cache.

For each request the scheduler matches the prompt in the radix tree, locks the
matched node (reference counter), allocates slots for what is missing
(evicting ``needed`` tokens and retrying once when the pool is short),
and, once the request finishes, inserts the full sequence and unlocks
(section 3, Algorithm 1).  ``plan_batch`` admits a batch of extend requests
(cached prefix P plus E new tokens) and decode requests (L - 1 cached tokens
plus one new token) and returns the per-request slot rows the kernels read
through ``req_to_token``.  A request whose context is not fully cached gets
slots for the missing part inserted first, standing in for the prefill that
produced it earlier.

Every tree and pool operation runs in the native library; this module only
sequences the calls and lays out the tables.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import OutOfSlots, RadixCache


@dataclass
class BatchPlan:
    rows: list[np.ndarray]           # slot of every position of each request
    ctx_lens: list[int]              # positions cached before the batch runs
    new_ctx: list[tuple[int, int]]   # [start, end) of context inserted for the batch
    matched: list[int]               # cached prompt tokens found by the first match
    locks: list[int] = field(default_factory=list)

    @property
    def hit_rate(self) -> float:
        tot = sum(self.ctx_lens)
        return float(sum(self.matched)) / tot if tot else 0.0


class Scheduler:
    def __init__(self, pool_slots: int, free_order=None):
        self.cache = RadixCache(pool_slots, free_order)
        self.ops = 0

    def alloc_or_evict(self, n: int) -> np.ndarray:
        self.ops += 1
        try:
            return self.cache.alloc(n)
        except OutOfSlots:
            self.ops += 2
            self.cache.evict(n)
            return self.cache.alloc(n)

    def finish_request(self, tokens) -> None:
        """A request that runs and finishes at once."""
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        node, m, slots = self.cache.match_prefix(t)
        self.cache.inc_ref(node)
        new = self.alloc_or_evict(t.shape[0] - m)
        self.cache.insert(t, np.concatenate([slots, new]))
        self.cache.dec_ref(node)
        self.ops += 4

    def admit(self, ctx, n_new: int):
        ctx = np.ascontiguousarray(ctx, dtype=np.int32)
        node, m, slots = self.cache.match_prefix(ctx)
        self.cache.inc_ref(node)
        self.ops += 2
        filled = (m, m)
        if m < ctx.shape[0]:
            new = self.alloc_or_evict(ctx.shape[0] - m)
            slots = np.concatenate([slots, new])
            _, node2 = self.cache.insert(ctx, slots)
            self.cache.inc_ref(node2)
            self.cache.dec_ref(node)
            self.ops += 3
            node = node2
            filled = (m, ctx.shape[0])
        own = self.alloc_or_evict(n_new)
        return node, m, np.concatenate([slots, own]).astype(np.int32), filled

    def plan_batch(self, extend, decode) -> BatchPlan:
        """extend: [(tokens, P, E)], decode: [(tokens, L)]; extends first."""
        plan = BatchPlan([], [], [], [])
        reqs = [(t, p, e) for t, p, e in extend] + [(t, l - 1, 1) for t, l in decode]
        for toks, c, k in reqs:
            node, m, row, filled = self.admit(np.asarray(toks)[:c], k)
            plan.rows.append(row)
            plan.ctx_lens.append(c)
            plan.new_ctx.append(filled)
            plan.matched.append(m)
            plan.locks.append(node)
        return plan

    def finish_batch(self, extend, decode, plan: BatchPlan) -> None:
        seqs = [np.asarray(t)[: p + e] for t, p, e in extend] + [np.asarray(t)[:l] for t, l in decode]
        for toks, row, node in zip(seqs, plan.rows, plan.locks):
            self.cache.insert(toks, row)
            self.cache.dec_ref(node)
            self.ops += 2


def build_table(rows: list[np.ndarray], stride: int | None = None, row_order=None):
    """Lays rows into req_to_token [R, stride] (int32, unused entries -1).

    Request r uses table row ``req_pool_idx[r]``; ``row_order`` permutes which
    table row each request gets (identity by default).
    """
    n = len(rows)
    stride = max((len(r) for r in rows), default=1) if stride is None else stride
    order = np.arange(n, dtype=np.int32) if row_order is None else np.asarray(row_order, dtype=np.int32)
    table = np.full((max(n, 1), max(stride, 1)), -1, dtype=np.int32)
    for r, row in enumerate(rows):
        table[order[r], : len(row)] = row
    return table, order
