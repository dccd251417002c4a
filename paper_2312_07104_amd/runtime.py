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

``CacheAwareScheduler`` is Algorithm 1's admission loop (cache-aware,
longest-shared-prefix-first scheduling with continuous batching, section 3 and
Appendix A.2), and ``run_offline`` processes a fixed batch one request at a
time in a chosen order, the setting of Theorem 3.1 (Appendix A.3), with
hit-rate accounting.

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


# ---- cache-aware scheduling (Algorithm 1, Theorem 3.1) ------------------------

POLICIES = ("lspf", "fcfs", "random")


@dataclass
class Request:
    """A request of the scheduler: prefill tokens plus a number of tokens it
    will generate (their slots are reserved at admission)."""
    rid: int
    tokens: np.ndarray
    out_len: int = 0
    node: int = 0
    prefix_len: int = 0
    prefix_slots: np.ndarray | None = None
    slots: np.ndarray | None = None

    def size(self) -> int:
        return int(self.tokens.shape[0]) + self.out_len


def _order(policy: str, items: list, keys: list[int], rng) -> list:
    """Longest matched prefix first (ties keep submission order), submission
    order, or a seeded random order."""
    if policy == "lspf":
        idx = sorted(range(len(items)), key=lambda i: -keys[i])
    elif policy == "fcfs":
        idx = list(range(len(items)))
    elif policy == "random":
        idx = list(rng.permutation(len(items)))
    else:
        raise ValueError(f"unknown policy {policy!r}; one of {POLICIES}")
    return [items[i] for i in idx]


class CacheAwareScheduler:
    """Algorithm 1: match every waiting request, sort by matched prefix length,
    admit requests while ``size + current_size < available_size`` (locking each
    admitted prefix lowers the available size by the tokens that stop being
    evictable), allocate the new tokens' slots for the admitted requests
    (evicting the needed size and retrying once when the pool is short), and on
    completion unlock the prefix and insert the finished sequence.

    ``current_size`` grows by each admitted request's size; the printed
    pseudocode never updates it (reading 6 of the design notes).  Counters:
    ``prefill_tokens`` (prompt tokens of admitted requests) and
    ``cached_prefill_tokens`` (of those, found in the cache at admission);
    ``hit_rate`` is their ratio.
    """

    def __init__(self, pool_slots: int, free_order=None, policy: str = "lspf", seed: int = 0):
        if policy not in POLICIES:
            raise ValueError(f"unknown policy {policy!r}; one of {POLICIES}")
        self.cache = RadixCache(pool_slots, free_order)
        self.policy = policy
        self.rng = np.random.default_rng(seed)
        self.waiting: list[Request] = []
        self.running: list[Request] = []
        self.prefill_tokens = 0
        self.cached_prefill_tokens = 0
        self._next_id = 0

    @property
    def hit_rate(self) -> float:
        return self.cached_prefill_tokens / self.prefill_tokens if self.prefill_tokens else 0.0

    def submit(self, tokens, out_len: int = 0) -> Request:
        r = Request(self._next_id, np.ascontiguousarray(tokens, dtype=np.int32), int(out_len))
        self._next_id += 1
        self.waiting.append(r)
        return r

    def schedule(self) -> list[Request]:
        """One pass of the admission loop; returns the requests admitted, each
        with ``slots`` covering its prompt and reserved output positions."""
        reqs = self.waiting
        for r in reqs:
            r.node, r.prefix_len, r.prefix_slots = self.cache.match_prefix(r.tokens)
        ordered = _order(self.policy, reqs, [r.prefix_len for r in reqs], self.rng)
        available = self.cache.evictable_size() + self.cache.available_size()
        current = 0
        batch = []
        for r in ordered:
            if r.size() + current < available:
                batch.append(r)
                available += self.cache.inc_ref(r.node)
                current += r.size()
        chosen = {r.rid for r in batch}
        self.waiting = [r for r in reqs if r.rid not in chosen]
        needed = sum(r.size() - r.prefix_len for r in batch)
        if needed:
            try:
                buf = self.cache.alloc(needed)
            except OutOfSlots:
                self.cache.evict(needed)
                buf = self.cache.alloc(needed)
        else:
            buf = np.empty(0, dtype=np.int32)
        off = 0
        for r in batch:
            k = r.size() - r.prefix_len
            r.slots = np.concatenate([r.prefix_slots, buf[off: off + k]]).astype(np.int32)
            off += k
            self.prefill_tokens += int(r.tokens.shape[0])
            self.cached_prefill_tokens += r.prefix_len
        self.running.extend(batch)
        return batch

    def finish(self, r: Request, generated=None) -> None:
        """Unlock the request's prefix and insert prompt + generated tokens with
        their slots; unused reserved slots go back to the pool."""
        gen = np.zeros(0, dtype=np.int32) if generated is None else np.ascontiguousarray(generated, dtype=np.int32)
        if gen.shape[0] > r.out_len:
            raise ValueError("more generated tokens than reserved")
        seq = np.concatenate([r.tokens, gen])
        used = seq.shape[0]
        self.cache.dec_ref(r.node)
        self.cache.insert(seq, r.slots[:used])
        if used < r.slots.shape[0]:
            self.cache.free_slots(r.slots[used:])
        self.running = [x for x in self.running if x.rid != r.rid]


@dataclass
class OfflineResult:
    order: list[int]          # request indices in processing order
    computed_tokens: int      # prefill tokens whose KV had to be computed
    prefill_tokens: int

    @property
    def hit_rate(self) -> float:
        return 1.0 - self.computed_tokens / self.prefill_tokens if self.prefill_tokens else 0.0


def run_offline(sequences, pool_slots: int, policy: str = "lspf", seed: int = 0, free_order=None) -> OfflineResult:
    """Processes a fixed batch one request at a time (Theorem 3.1's setting):
    pick the next request by the policy (for ``lspf``, the one whose prompt
    has the longest cached prefix right now), lock its cached prefix, compute
    (allocate) the rest, insert, unlock.  Returns the order and the number of
    computed tokens, which for ``lspf`` with ``pool_slots`` at least the longest
    request equals the number of tokens on the edges of the batch's radix
    tree."""
    if policy not in POLICIES:
        raise ValueError(f"unknown policy {policy!r}; one of {POLICIES}")
    seqs = [np.ascontiguousarray(s, dtype=np.int32) for s in sequences]
    cache = RadixCache(pool_slots, free_order)
    rng = np.random.default_rng(seed)
    remaining = list(range(len(seqs)))
    if policy == "random":
        remaining = [remaining[i] for i in rng.permutation(len(remaining))]
    order, computed, total = [], 0, 0
    while remaining:
        if policy == "lspf":
            lens = [cache.match_prefix(seqs[i])[1] for i in remaining]
            k = max(range(len(remaining)), key=lambda j: (lens[j], -j))
        else:
            k = 0
        i = remaining.pop(k)
        node, m, slots = cache.match_prefix(seqs[i])
        cache.inc_ref(node)
        need = seqs[i].shape[0] - m
        if need:
            try:
                new = cache.alloc(need)
            except OutOfSlots:
                cache.evict(need)
                new = cache.alloc(need)
            cache.insert(seqs[i], np.concatenate([slots, new]))
        cache.dec_ref(node)
        order.append(i)
        computed += need
        total += int(seqs[i].shape[0])
    return OfflineResult(order, computed, total)


# ---------------------------------------------------------------------------
# Data parallelism: a router meta-tree over replica workers (Appendix A.4)
# ---------------------------------------------------------------------------

DP_POLICIES = ("affinity", "least_loaded", "round_robin", "random")


@dataclass
class DataParallelResult:
    policy: str
    n_workers: int
    prefill_tokens: int
    computed_tokens: int
    worker_work: list[int]         # computed (prefilled) tokens per worker
    worker_requests: list[int]
    router_nodes: int

    @property
    def hit_rate(self) -> float:
        return 1.0 - self.computed_tokens / self.prefill_tokens if self.prefill_tokens else 0.0

    @property
    def imbalance(self) -> float:
        """Largest worker's work over the mean (1.0 = perfectly balanced)."""
        mean = sum(self.worker_work) / len(self.worker_work)
        return max(self.worker_work) / mean if mean else 1.0


def _serve(cache: RadixCache, seq: np.ndarray) -> int:
    """One request on one worker: match, lock, compute (allocate) the rest,
    evicting when the pool is short (Algorithm 1), insert, unlock.  Returns
    the number of computed tokens."""
    node, m, slots = cache.match_prefix(seq)
    cache.inc_ref(node)
    need = seq.shape[0] - m
    if need:
        try:
            new = cache.alloc(need)
        except OutOfSlots:
            cache.evict(need)
            new = cache.alloc(need)
        cache.insert(seq, np.concatenate([slots, new]))
    cache.dec_ref(node)
    return need


def run_data_parallel(sequences, n_workers: int, pool_slots: int, policy: str = "affinity",
                      commit_every: int = 1, slack: float = 0.1, seed: int = 0, free_order=None,
                      probe=None) -> DataParallelResult:
    """Dispatches a request stream over ``n_workers`` replicas, each with its
    own radix cache of ``pool_slots`` slots, through the router meta-tree.

    The router records a request's sequence for the chosen worker at dispatch
    (both sides update their trees independently); workers log their
    evictions and the router applies the logs every ``commit_every`` requests
    (its idle periods), so in between its view may be stale.

    Policies: ``affinity`` picks the worker with the longest cached prefix of
    the prompt (router view) among the workers whose accumulated work is
    within ``slack`` of the mean plus this request (ties and no match: the
    least loaded); ``least_loaded``, ``round_robin`` and ``random`` ignore
    the caches.  ``probe(router, workers)`` is called after every commit
    (tests check the router against the worker trees there)."""
    if policy not in DP_POLICIES:
        raise ValueError(f"unknown policy {policy!r}; one of {DP_POLICIES}")
    if n_workers < 1 or commit_every < 1 or slack < 0:
        raise ValueError("n_workers and commit_every must be >= 1 and slack >= 0")
    from . import Router

    seqs = [np.ascontiguousarray(s, dtype=np.int32) for s in sequences]
    router = Router(n_workers)
    workers = [RadixCache(pool_slots, free_order) for _ in range(n_workers)]
    for c in workers:
        c.log_evictions(True)
    rng = np.random.default_rng(seed)
    work = [0] * n_workers
    nreq = [0] * n_workers
    computed = total = 0

    def commit():
        for w, c in enumerate(workers):
            while True:
                e = c.pop_eviction()
                if e is None:
                    break
                router.evict(w, e[0], e[1])
        if probe is not None:
            probe(router, workers)

    for i, seq in enumerate(seqs):
        n = int(seq.shape[0])
        if policy == "affinity":
            m = router.match(seq)
            mean = sum(work) / n_workers
            ok = [w for w in range(n_workers) if work[w] <= (1.0 + slack) * mean + n] or list(range(n_workers))
            w = max(ok, key=lambda x: (int(m[x]), -work[x], -x))
        elif policy == "least_loaded":
            w = min(range(n_workers), key=lambda x: (work[x], x))
        elif policy == "round_robin":
            w = i % n_workers
        else:
            w = int(rng.integers(n_workers))
        router.insert(w, seq)
        need = _serve(workers[w], seq)
        work[w] += need
        nreq[w] += 1
        computed += need
        total += n
        if (i + 1) % commit_every == 0:
            commit()
    commit()
    return DataParallelResult(policy, n_workers, total, computed, work, nreq, router.num_nodes())
