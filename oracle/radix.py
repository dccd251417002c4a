"""Radix tree over token sequences and the shared token pool, in plain Python.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Follows section 3 of the paper (RadixAttention) and Algorithm 1 (cache-aware
scheduling with continuous batching):

* edges carry runs of tokens; the tree maps token sequences to the pool slots
  holding their KV entries, one slot per token (pages of one token);
* a reference counter per node counts the running requests using it; a node
  is evictable when its counter is zero (``evictable_size`` sums the tokens of
  such nodes);
* eviction removes the least recently used leaf first; a parent left without
  children becomes a leaf and may be evicted next;
* cached tokens and running requests share one pool with no fixed partition.

Where the paper is silent this file takes these readings (each side of the
parity tests implements the same ones):

1. "Used" means touched by ``match_prefix`` or ``insert``: every call bumps a
   logical clock once and stamps every node on the path it walks.
2. Eviction picks the evictable leaf with the smallest (stamp, node id); it
   frees whole leaves, so it may free more than asked, and stops early when
   nothing is evictable.  Nodes are never merged back.
3. ``match_prefix`` splits an edge where the match ends inside it, so the
   returned node covers exactly the matched prefix; ``insert`` splits where a
   new sequence diverges inside an edge.  A split keeps the old node id for
   the lower part and gives the new upper node the next id, the old node's
   reference count and its stamp.
4. A reference lock covers the whole root-to-node path.  ``inc_ref`` returns
   minus the tokens that stopped being evictable, ``dec_ref`` plus the tokens
   that became evictable (underflow is an error and changes nothing).
5. ``insert`` keeps already cached slots; a caller slot that differs from the
   cached slot at the same position goes back to the pool, in position order.
6. The pool is a FIFO queue of free slots with a caller-given initial order;
   ``alloc(n)`` pops n slots from the front or fails with no effect; ``free``
   appends in the given order and rejects slots out of range or already free.
"""
from __future__ import annotations

from collections import deque


class RadixError(Exception):
    pass


class OutOfSlots(RadixError):
    pass


class _Node:
    __slots__ = ("id", "parent", "key", "slots", "children", "ref", "stamp")

    def __init__(self, nid, parent, key, slots, ref, stamp):
        self.id = nid
        self.parent = parent
        self.key = list(key)
        self.slots = list(slots)
        self.children = {}
        self.ref = ref
        self.stamp = stamp


class RadixCache:
    """Radix tree plus slot pool (the paper's T and P, sharing accounting)."""

    def __init__(self, pool_slots: int, free_order=None):
        if pool_slots < 0:
            raise RadixError("pool size must be non-negative")
        order = list(range(pool_slots)) if free_order is None else [int(x) for x in free_order]
        if sorted(order) != list(range(pool_slots)):
            raise RadixError("initial free order must be a permutation of the pool")
        self.pool_slots = pool_slots
        self.free = deque(order)
        self.is_free = [True] * pool_slots
        self.root = _Node(0, None, [], [], 0, 0)
        self.nodes = {0: self.root}
        self.next_id = 1
        self.clock = 0

    # ---- pool ---------------------------------------------------------------
    def alloc(self, n: int) -> list[int]:
        if n < 0:
            raise RadixError("negative allocation")
        if n > len(self.free):
            raise OutOfSlots(n)
        out = [self.free.popleft() for _ in range(n)]
        for s in out:
            self.is_free[s] = False
        return out

    def free_slots(self, slots) -> None:
        slots = [int(s) for s in slots]
        seen = set()
        for s in slots:
            if not 0 <= s < self.pool_slots or self.is_free[s] or s in seen:
                raise RadixError(f"slot {s} is out of range or already free")
            seen.add(s)
        for s in slots:
            self.is_free[s] = True
            self.free.append(s)

    def available_size(self) -> int:
        return len(self.free)

    # ---- tree ---------------------------------------------------------------
    def _split(self, x: _Node, c: int) -> _Node:
        y = _Node(self.next_id, x.parent, x.key[:c], x.slots[:c], x.ref, x.stamp)
        self.next_id += 1
        self.nodes[y.id] = y
        x.parent.children[y.key[0]] = y
        x.key, x.slots = x.key[c:], x.slots[c:]
        x.parent = y
        y.children[x.key[0]] = x
        return y

    @staticmethod
    def _common(a: list[int], b: list[int]) -> int:
        n = min(len(a), len(b))
        i = 0
        while i < n and a[i] == b[i]:
            i += 1
        return i

    def _walk(self, tokens: list[int], on_match=None):
        """Descend along ``tokens``, splitting where the match ends mid-edge."""
        self.clock += 1
        node, pos = self.root, 0
        while pos < len(tokens):
            child = node.children.get(tokens[pos])
            if child is None:
                break
            c = self._common(child.key, tokens[pos:])
            if c < len(child.key):
                child = self._split(child, c)
            child.stamp = self.clock
            if on_match is not None:
                on_match(child, pos)
            pos += c
            node = child
        return node, pos

    def match_prefix(self, tokens):
        """Longest cached prefix: (node id, matched length, its slots)."""
        tokens = [int(t) for t in tokens]
        slots: list[int] = []
        node, pos = self._walk(tokens, lambda ch, p: slots.extend(ch.slots))
        return node.id, pos, slots

    def insert(self, tokens, slots):
        """Cache ``tokens`` -> ``slots``; returns (already cached length, node id)."""
        tokens = [int(t) for t in tokens]
        slots = [int(s) for s in slots]
        if len(tokens) != len(slots):
            raise RadixError("tokens and slots differ in length")
        dup: list[int] = []

        def keep_cached(ch, p):
            for i, s in enumerate(ch.slots):
                if slots[p + i] != s:
                    dup.append(slots[p + i])

        node, pos = self._walk(tokens, keep_cached)
        cached = pos
        if dup:
            self.free_slots(dup)
        if pos < len(tokens):
            leaf = _Node(self.next_id, node, tokens[pos:], slots[pos:], 0, self.clock)
            self.next_id += 1
            self.nodes[leaf.id] = leaf
            node.children[tokens[pos]] = leaf
            node = leaf
        return cached, node.id

    def _path(self, nid: int):
        if nid not in self.nodes:
            raise RadixError(f"unknown node {nid}")
        x = self.nodes[nid]
        while x is not self.root:
            yield x
            x = x.parent

    def inc_ref(self, nid: int) -> int:
        delta = 0
        for x in self._path(nid):
            if x.ref == 0:
                delta -= len(x.key)
            x.ref += 1
        return delta

    def dec_ref(self, nid: int) -> int:
        path = list(self._path(nid))
        if any(x.ref == 0 for x in path):
            raise RadixError("reference counter underflow")
        delta = 0
        for x in path:
            x.ref -= 1
            if x.ref == 0:
                delta += len(x.key)
        return delta

    def evict(self, n_tokens: int) -> tuple[int, list[int]]:
        """Free at least n_tokens by evicting LRU unreferenced leaves."""
        freed: list[int] = []
        while len(freed) < n_tokens:
            cands = [x for x in self.nodes.values()
                     if x is not self.root and x.ref == 0 and not x.children]
            if not cands:
                break
            x = min(cands, key=lambda n: (n.stamp, n.id))
            del x.parent.children[x.key[0]]
            del self.nodes[x.id]
            freed.extend(x.slots)
            self.free_slots(x.slots)
        return len(freed), freed

    def evictable_size(self) -> int:
        return sum(len(x.key) for x in self.nodes.values() if x is not self.root and x.ref == 0)

    def cached_tokens(self) -> int:
        return sum(len(x.key) for x in self.nodes.values())

    def snapshot(self) -> dict:
        """Canonical state: nodes by id, the free queue and the clock."""
        nodes = []
        for nid in sorted(self.nodes):
            x = self.nodes[nid]
            nodes.append((nid, -1 if x.parent is None else x.parent.id, x.ref, x.stamp,
                          tuple(x.key), tuple(x.slots)))
        return {"nodes": nodes, "free": list(self.free), "clock": self.clock}
