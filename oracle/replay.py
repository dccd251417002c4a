"""Algorithm 1's per-request call sequence, run on the oracle radix tree.

TEST INFRASTRUCTURE ONLY (see the package docstring).

For every request the scheduler of Algorithm 1 matches the prompt against the
tree, locks the matched node, allocates pool slots for what is missing
(evicting ``needed`` tokens and retrying once if the pool is short), runs the
batch, and on completion inserts the finished sequence and releases the lock.
This module replays a ``workload.scenarios.Scenario`` that way:

* history requests finish at once (match, lock, allocate, insert, unlock);
* a phase admits its extend requests, then its decode requests, in order.  A
  request's context (the P prefix tokens of an extend, the first L-1 tokens
  of a decode) must be cached before attention runs: whatever the match does
  not find is allocated and inserted first, standing in for an earlier prefill
  of those tokens, and the request then holds a lock on the whole context.
  The request's own new tokens (E, or 1 for decode) get fresh slots;
* after the phase runs, each request inserts its full sequence and unlocks.

The output per phase is the slot table: row r lists the slot of every
position of request r.
"""
from __future__ import annotations

from dataclasses import dataclass, field

from .radix import OutOfSlots, RadixCache


@dataclass
class PhaseTables:
    rows: list[list[int]]            # slot of every position, per request
    ctx_lens: list[int]              # positions that are context (cached before the phase)
    new_ctx: list[tuple[int, int]]   # per request: [start, end) of context filled this phase
    matched: list[int]               # cached prompt tokens found by the first match
    locks: list[int] = field(default_factory=list)


class Replayer:
    def __init__(self, pool_slots: int, free_order=None):
        self.tree = RadixCache(pool_slots, free_order)
        self.ops = 0

    def _op(self, name, *args):
        self.ops += 1
        return getattr(self.tree, name)(*args)

    def alloc_or_evict(self, n: int) -> list[int]:
        try:
            return self._op("alloc", n)
        except OutOfSlots:
            self._op("evict", n)
            return self._op("alloc", n)

    def finish_request(self, tokens) -> None:
        """A request that runs and finishes at once (history traffic)."""
        nid, m, slots = self._op("match_prefix", tokens)
        self._op("inc_ref", nid)
        new = self.alloc_or_evict(len(tokens) - m)
        self._op("insert", tokens, slots + new)
        self._op("dec_ref", nid)

    def admit(self, ctx, n_new: int):
        nid, m, slots = self._op("match_prefix", ctx)
        self._op("inc_ref", nid)
        filled = (m, m)
        if m < len(ctx):
            new = self.alloc_or_evict(len(ctx) - m)
            _, nid2 = self._op("insert", ctx, slots + new)
            self._op("inc_ref", nid2)
            self._op("dec_ref", nid)
            nid = nid2
            slots = slots + new
            filled = (m, len(ctx))
        own = self.alloc_or_evict(n_new)
        return nid, m, slots + own, filled

    def run_phase(self, phase) -> PhaseTables:
        t = PhaseTables([], [], [], [])
        reqs = [(r.tokens, r.prefix_len, r.extend_len) for r in phase.extend]
        reqs += [(r.tokens, r.seq_len - 1, 1) for r in phase.decode]
        for toks, c, k in reqs:
            nid, m, row, filled = self.admit(list(toks[:c]), k)
            t.rows.append(row)
            t.ctx_lens.append(c)
            t.new_ctx.append(filled)
            t.matched.append(m)
            t.locks.append(nid)
        return t

    def finish_phase(self, phase, t: PhaseTables) -> None:
        seqs = [r.tokens[: r.prefix_len + r.extend_len] for r in phase.extend]
        seqs += [r.tokens[: r.seq_len] for r in phase.decode]
        for toks, row, nid in zip(seqs, t.rows, t.locks):
            self._op("insert", list(toks), row)
            self._op("dec_ref", nid)


def replay(scenario, history_limit: int | None = None):
    """Replay history and every phase; returns (replayer, [PhaseTables])."""
    rp = Replayer(scenario.pool_slots, scenario.free_order())
    n_hist = scenario.history_len if history_limit is None else min(history_limit, scenario.history_len)
    for i in range(n_hist):
        rp.finish_request(list(scenario.history(i)))
    tables = []
    for ph in scenario.phases:
        t = rp.run_phase(ph)
        tables.append(t)
        rp.finish_phase(ph, t)
    return rp, tables
