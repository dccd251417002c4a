"""Pins for the oracle radix tree and token pool (CPU only).

* A brute-force model (a dict from every cached token prefix to its slot)
  must agree with every match the tree answers, through random inserts,
  locks and evictions on tiny alphabets.
* Invariants: reference counts equal the number of locks covering a node,
  evictable_size sums unreferenced tokens, pool slots are conserved.
* The nine-step RadixAttention example of section 3 (chat sessions, few-shot
  queries, self-consistency sampling) is scripted with a pool size that
  forces the evictions the paper narrates.  The figure itself is not in the
  text, so node labels cannot be checked, only the structure and which
  sessions get evicted: parity partially pinned.
"""
import numpy as np
import pytest

from oracle.radix import OutOfSlots, RadixCache, RadixError
from oracle.replay import Replayer, replay
from workload import scenarios as S


# ------------------------------------------------------------ helpers -------

def finish(t: RadixCache, seq):
    """Algorithm 1 for one request that finishes at once."""
    nid, m, slots = t.match_prefix(seq)
    t.inc_ref(nid)
    need = len(seq) - m
    try:
        new = t.alloc(need)
    except OutOfSlots:
        t.evict(need)
        new = t.alloc(need)
    t.insert(seq, slots + new)
    t.dec_ref(nid)


def leaves(t):
    return sorted(tuple(x.key) for x in t.nodes.values() if x is not t.root and not x.children)


def edge_keys(t):
    return sorted(tuple(x.key) for x in t.nodes.values() if x is not t.root)


def check_invariants(t: RadixCache, locks: list[int], held: int = 0):
    nodes = [x for x in t.nodes.values() if x is not t.root]
    # reference counts equal the locks whose root path covers the node
    cover = {x.id: 0 for x in nodes}
    for nid in locks:
        for x in t._path(nid):
            cover[x.id] += 1
    for x in nodes:
        assert x.ref == cover[x.id]
        assert len(x.key) == len(x.slots) > 0
        assert x.parent.children[x.key[0]] is x
    assert t.evictable_size() == sum(len(x.key) for x in nodes if x.ref == 0)
    tree_slots = [s for x in nodes for s in x.slots]
    assert len(set(tree_slots)) == len(tree_slots)
    assert not (set(tree_slots) & set(t.free))
    assert len(tree_slots) + len(t.free) + held == t.pool_slots
    for s in range(t.pool_slots):
        assert t.is_free[s] == (s in set(t.free))


# ---------------------------------------------------- brute-force model -----

class Model:
    def __init__(self):
        self.m = {}

    def insert(self, seq, slots):
        for i in range(len(seq)):
            self.m.setdefault(tuple(seq[: i + 1]), slots[i])

    def evicted(self, freed):
        fs = set(freed)
        self.m = {k: s for k, s in self.m.items() if s not in fs}

    def match(self, seq):
        n = 0
        while n < len(seq) and tuple(seq[: n + 1]) in self.m:
            n += 1
        return n, [self.m[tuple(seq[: i + 1])] for i in range(n)]


@pytest.mark.parametrize("seed", range(12))
def test_matches_brute_force_model(seed):
    rng = np.random.default_rng(seed)
    alpha = int(rng.integers(2, 5))
    pool = int(rng.integers(8, 33))
    t = RadixCache(pool, rng.permutation(pool))
    model = Model()
    locks: list[int] = []
    held = 0
    for _ in range(300):
        seq = [int(x) for x in rng.integers(0, alpha, size=int(rng.integers(1, 13)))]
        op = rng.random()
        if op < 0.45:  # cache a sequence (a request that finished)
            nid, m, slots = t.match_prefix(seq)
            assert (m, slots) == model.match(seq)
            t.inc_ref(nid)
            need = len(seq) - m
            try:
                new = t.alloc(need)
            except OutOfSlots:
                _, freed = t.evict(need)
                model.evicted(freed)
                try:
                    new = t.alloc(need)
                except OutOfSlots:
                    t.dec_ref(nid)
                    continue
            t.insert(seq, slots + new)
            model.insert(seq, slots + new)
            t.dec_ref(nid)
        elif op < 0.65:  # lock a matched prefix
            nid, m, slots = t.match_prefix(seq)
            assert (m, slots) == model.match(seq)
            if nid != 0:
                t.inc_ref(nid)
                locks.append(nid)
        elif op < 0.8 and locks:  # release a lock
            t.dec_ref(locks.pop(int(rng.integers(len(locks)))))
        elif op < 0.9:
            _, freed = t.evict(int(rng.integers(0, 6)))
            model.evicted(freed)
        else:  # a running request holds fresh slots, then returns them
            n = int(rng.integers(0, 4))
            if n <= t.available_size():
                s = t.alloc(n)
                held += n
                check_invariants(t, locks, held)
                t.free_slots(s)
                held -= n
        check_invariants(t, locks, held)
    # every cached path is found in full
    for x in list(t.nodes.values()):
        path, y = [], x
        while y is not t.root:
            path = y.key + path
            y = y.parent
        assert t.match_prefix(path)[1] == len(path)


# ---------------------------------------------------- section 3 figure ------

def run(start, n):
    return list(range(start, start + n))


def test_nine_step_example():
    SYS, T1, T2 = run(1, 8), run(100, 4), run(200, 16)
    V1, V2 = run(300, 4), run(400, 16)
    FS, Q1, Q2, Q3 = run(500, 6), run(600, 3), run(700, 3), run(800, 3)
    T3 = run(900, 18)
    SMP = [run(1000 + 10 * k, 4) for k in range(3)]
    t = RadixCache(47)
    # (1) empty
    assert edge_keys(t) == []
    # (2) first chat turn: one edge from the root
    finish(t, SYS + T1)
    assert edge_keys(t) == [tuple(SYS + T1)]
    # (3) second turn reuses the first and is appended as a new node
    finish(t, SYS + T1 + T2)
    assert edge_keys(t) == sorted([tuple(SYS + T1), tuple(T2)])
    # (4) a second session splits the first edge to share the system prompt
    finish(t, SYS + V1)
    assert edge_keys(t) == sorted([tuple(SYS), tuple(T1), tuple(T2), tuple(V1)])
    # (5) memory is short: the least recently used leaf (session 1's second
    # turn) is evicted; the new turn hangs under session 2's node
    finish(t, SYS + V1 + V2)
    assert edge_keys(t) == sorted([tuple(SYS), tuple(T1), tuple(V1), tuple(V2)])
    # (6) a few-shot query shares nothing: a new branch at the root
    finish(t, FS + Q1)
    assert tuple(FS + Q1) in edge_keys(t)
    # (7) more queries with the same examples split the few-shot edge
    finish(t, FS + Q2)
    finish(t, FS + Q3)
    assert {tuple(FS), tuple(Q1), tuple(Q2), tuple(Q3)} <= set(edge_keys(t))
    # (8) session 1 returns; session 2's two nodes are the LRU ones and go
    finish(t, SYS + T1 + T3)
    keys = set(edge_keys(t))
    assert tuple(V1) not in keys and tuple(V2) not in keys
    assert {tuple(SYS), tuple(T1), tuple(T3), tuple(FS), tuple(Q1), tuple(Q2), tuple(Q3)} <= keys
    # (9) self-consistency samples for one question evict three nodes
    before = set(edge_keys(t))
    for s in SMP:
        finish(t, FS + Q3 + s)
    gone = before - set(edge_keys(t))
    assert gone == {tuple(Q1), tuple(Q2), tuple(T3)}
    assert {tuple(s) for s in SMP} <= set(edge_keys(t))
    check_invariants(t, [])


# ------------------------------------------------------- hand examples ------

def test_lru_order_and_tie_break():
    t = RadixCache(12)
    for seq in ([1, 2], [3, 4], [5, 6]):
        finish(t, seq)
    t.match_prefix([3, 4])  # touch [3, 4]: now [1, 2] then [5, 6] are older
    n, freed = t.evict(3)
    assert n == 4 and len(freed) == 4
    assert leaves(t) == [(3, 4)]


def test_parent_becomes_evictable_leaf():
    t = RadixCache(10)
    finish(t, [1, 2, 3])
    finish(t, [1, 2, 3, 4, 5])
    finish(t, [9])
    t.match_prefix([9])
    # leaf [4, 5] goes first; its parent [1, 2, 3] is then the oldest leaf
    n, _ = t.evict(4)
    assert n == 5 and leaves(t) == [(9,)]


def test_locked_nodes_survive_eviction():
    t = RadixCache(6)
    finish(t, [1, 2, 3])
    nid, m, _ = t.match_prefix([1, 2, 3])
    assert t.inc_ref(nid) == -3
    assert t.evict(10) == (0, [])
    assert t.dec_ref(nid) == 3
    assert t.evict(1)[0] == 3


def test_split_keeps_lower_id_and_copies_ref():
    t = RadixCache(10)
    finish(t, [1, 2, 3, 4])
    nid, _, _ = t.match_prefix([1, 2, 3, 4])
    t.inc_ref(nid)
    up, m, slots = t.match_prefix([1, 2, 7])
    assert m == 2 and up != nid and t.nodes[nid].key == [3, 4]
    assert t.nodes[up].ref == 1 and t.nodes[nid].parent.id == up
    assert t.dec_ref(nid) == 4  # both halves become evictable


def test_insert_frees_only_differing_duplicates():
    t = RadixCache(8, [7, 6, 5, 4, 3, 2, 1, 0])
    finish(t, [1, 2, 3])                   # slots 7 6 5
    a = t.alloc(3)                         # 4 3 2
    cached, _ = t.insert([1, 2, 3, 9], [7] + a)
    assert cached == 3
    # slots [7, 4, 3, 2]: 7 is the cached slot, 4 and 3 duplicate cached
    # positions and go back to the pool, 2 becomes token 9's slot
    assert list(t.free) == [1, 0, 4, 3]


def test_errors_change_nothing():
    t = RadixCache(4)
    finish(t, [1, 2])
    snap = t.snapshot()
    with pytest.raises(OutOfSlots):
        t.alloc(3)
    assert t.snapshot() == snap
    nid, _, _ = t.match_prefix([1, 2])
    snap = t.snapshot()
    with pytest.raises(RadixError):
        t.dec_ref(nid)
    with pytest.raises(RadixError):
        t.free_slots([3, 3])  # already free
    with pytest.raises(RadixError):
        t.free_slots([4])     # out of range
    with pytest.raises(RadixError):
        t.inc_ref(12345)      # unknown node
    assert t.snapshot() == snap
    assert t.alloc(0) == []


# --------------------------------------------------------------- replay -----

def test_replay_tables_cfg1():
    sc = S.cfg1_decode_tiny()
    rp, tables = replay(sc)
    t = tables[0]
    assert [len(r) for r in t.rows] == [r.seq_len for r in sc.phases[0].decode]
    # the 128-token shared prefix maps to the same slots in every row
    for r in t.rows[1:]:
        assert r[:128] == t.rows[0][:128]
    # every slot distinct within a row, all in range
    for r in t.rows:
        assert len(set(r)) == len(r) and all(0 <= s < sc.pool_slots for s in r)


def test_replay_mixed_small_conserves_pool():
    sc = S.cfg5_mixed_small()
    rp, tables = replay(sc)
    check_invariants(rp.tree, [])
    assert rp.ops > 5 * sc.history_len
