"""The data-parallel router's view of which worker holds which prefix, as
plain sets.  TEST INFRASTRUCTURE ONLY (see the package docstring).

Appendix A.4 of the paper: every replica worker keeps its own radix tree; a
router keeps a meta-tree that tracks the workers' trees, matches arriving
requests against it to dispatch by prefix affinity, records what it sends to
each worker, and applies the evictions workers commit to a queue.

Written as sets of prefixes instead of a tree, so a reader can check it by
eye: a worker's holding is the set of all non-empty prefixes (tuples) of the
sequences recorded for it.

* ``insert(w, seq)``: worker w now holds every prefix of seq.
* ``evict(w, path, k)``: worker w dropped the last k tokens of ``path``, a
  leaf of its tree, so it holds no prefix that passes through the first
  dropped position: every held prefix p with len(p) > len(path) - k and
  p[:len(path) - k + 1] == path[:len(path) - k + 1] goes.
* ``match(seq)[w]``: the length of the longest prefix of seq that w holds.
* ``held(w)``: how many token positions w holds (its number of prefixes).
"""
from __future__ import annotations


class BruteRouter:
    def __init__(self, n_workers: int):
        self.n_workers = n_workers
        self.sets: list[set] = [set() for _ in range(n_workers)]

    def insert(self, w: int, seq) -> None:
        s = tuple(int(t) for t in seq)
        for i in range(1, len(s) + 1):
            self.sets[w].add(s[:i])

    def evict(self, w: int, path, k: int) -> None:
        if k <= 0:
            return
        p = tuple(int(t) for t in path)
        head = p[: len(p) - k + 1]
        self.sets[w] = {q for q in self.sets[w] if not (len(q) >= len(head) and q[: len(head)] == head)}

    def match(self, seq) -> list[int]:
        s = tuple(int(t) for t in seq)
        out = []
        for w in range(self.n_workers):
            m = 0
            for i in range(1, len(s) + 1):
                if s[:i] in self.sets[w]:
                    m = i
                else:
                    break
            out.append(m)
        return out

    def held(self, w: int) -> int:
        return len(self.sets[w])
