"""The native library on the CPU: exported ABI, and the C++ radix cache bit-exact
against the oracle tree (no GPU needed; only host entry points are called)."""
import re
from pathlib import Path

import numpy as np
import pytest

ROOT = Path(__file__).resolve().parents[1]

pa = pytest.importorskip("paper_2312_07104_amd", reason="native library not built")
from paper_2312_07104_amd.runtime import Scheduler  # noqa: E402

from oracle import radix as orx  # noqa: E402
from oracle.replay import replay as oracle_replay  # noqa: E402
from workload import scenarios as S  # noqa: E402


def header_functions():
    text = (ROOT / "include" / "radixattn.h").read_text()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ra_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = header_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(pa._lib, n), n
    assert set(names) <= set(pa.EXPORTED) | {"ra_last_error"}


def _both(pool, order):
    return orx.RadixCache(pool, order), pa.RadixCache(pool, order)


@pytest.mark.parametrize("seed", range(16))
def test_random_ops_bit_exact(seed):
    rng = np.random.default_rng(100 + seed)
    alpha = int(rng.integers(2, 6))
    pool = int(rng.integers(6, 48))
    order = rng.permutation(pool).astype(np.int32)
    o, n = _both(pool, order)
    locks = []
    held = []
    for step in range(400):
        seq = [int(x) for x in rng.integers(0, alpha, size=int(rng.integers(1, 15)))]
        op = rng.random()
        if op < 0.3:
            a = o.match_prefix(seq)
            b = n.match_prefix(seq)
            assert (a[0], a[1], list(a[2])) == (b[0], b[1], b[2].tolist())
        elif op < 0.55:
            nid, m, slots = o.match_prefix(seq)
            n.match_prefix(seq)
            need = len(seq) - m
            if need <= o.available_size():
                s_o = o.alloc(need)
                s_n = n.alloc(need)
                assert s_o == s_n.tolist()
                # occasionally hand in a stale duplicate to exercise the free path
                full = list(slots) + s_o
                if m and rng.random() < 0.3 and o.available_size() >= 1:
                    dup = o.alloc(1)
                    n.alloc(1)
                    full[int(rng.integers(m))] = dup[0]
                assert o.insert(seq, full) == n.insert(seq, full)
        elif op < 0.7:
            nid, _, _ = o.match_prefix(seq)
            n.match_prefix(seq)
            if nid:
                assert o.inc_ref(nid) == n.inc_ref(nid)
                locks.append(nid)
        elif op < 0.8 and locks:
            nid = locks.pop(int(rng.integers(len(locks))))
            assert o.dec_ref(nid) == n.dec_ref(nid)
        elif op < 0.9:
            k = int(rng.integers(0, 8))
            assert o.evict(k)[0] == n.evict(k)
        else:
            k = int(rng.integers(0, 4))
            if k <= o.available_size():
                held.append(o.alloc(k))
                assert held[-1] == n.alloc(k).tolist()
            elif held:
                h = held.pop()
                o.free_slots(h)
                n.free_slots(h)
        assert o.snapshot() == n.snapshot()
        assert o.evictable_size() == n.evictable_size()
        assert o.available_size() == n.available_size()
        assert o.cached_tokens() == n.cached_tokens()


def test_errors_match_and_change_nothing():
    o, n = _both(5, None)
    for t in (o, n):
        t.insert([1, 2], t.alloc(2))
    nid, _, _ = n.match_prefix([1, 2])
    o.match_prefix([1, 2])
    snap = n.snapshot()
    with pytest.raises(pa.OutOfSlots):
        n.alloc(4)
    with pytest.raises(pa.RadixAttnError):
        n.dec_ref(nid)
    with pytest.raises(pa.RadixAttnError):
        n.free_slots([4, 4])
    with pytest.raises(pa.RadixAttnError):
        n.free_slots([7])
    with pytest.raises(pa.RadixAttnError):
        n.inc_ref(999)
    with pytest.raises(pa.RadixAttnError):
        n.insert([1, 2, 3], [0, 1, 99])  # new slot out of range
    assert n.snapshot() == snap == o.snapshot()
    with pytest.raises(pa.RadixAttnError):
        pa.RadixCache(3, [0, 0, 1])


def _native_replay(sc, history_limit=None):
    sch = Scheduler(sc.pool_slots, sc.free_order())
    n_hist = sc.history_len if history_limit is None else min(history_limit, sc.history_len)
    for i in range(n_hist):
        sch.finish_request(sc.history(i))
    plans = []
    for ph in sc.phases:
        ext = [(r.tokens, r.prefix_len, r.extend_len) for r in ph.extend]
        dec = [(r.tokens, r.seq_len) for r in ph.decode]
        p = sch.plan_batch(ext, dec)
        plans.append(p)
        sch.finish_batch(ext, dec, p)
    return sch, plans


@pytest.mark.parametrize("name", ["decode_tiny", "mixed_small", "branching_small"])
def test_scenario_tables_bit_exact(name):
    if name == "branching_small":
        sc = S.cfg4_branching(n_branch=6, root_len=300, branch_len=40, extend_len=9, pool=2048)
    else:
        sc = S.ALL[name]()
    rp, tables = oracle_replay(sc)
    sch, plans = _native_replay(sc)
    for t, p in zip(tables, plans):
        assert [list(r) for r in t.rows] == [r.tolist() for r in p.rows]
        assert t.new_ctx == p.new_ctx and t.matched == p.matched and t.locks == p.locks
    assert rp.tree.snapshot() == sch.cache.snapshot()


@pytest.mark.parametrize("seed", range(2))
def test_large_tree_bit_exact(seed):
    """Trees of thousands of edges (the child-edge table grows past its first
    sizes and deletes entries inside long probe runs on eviction), with many
    requests ending inside shared edges: match results after every call and
    whole-tree snapshots every 250 operations equal the oracle's."""
    rng = np.random.default_rng(7000 + seed)
    pool = 6000
    o, n = _both(pool, rng.permutation(pool).astype(np.int32))
    stems = [[int(x) for x in rng.integers(0, 40, size=int(rng.integers(20, 200)))] for _ in range(12)]
    for step in range(2500):
        stem = stems[int(rng.integers(len(stems)))]
        seq = stem[: int(rng.integers(1, len(stem) + 1))] + [int(x) for x in rng.integers(0, 40, size=int(rng.integers(0, 12)))]
        nid, m, slots = o.match_prefix(seq)
        b = n.match_prefix(seq)
        assert (nid, m, list(slots)) == (b[0], b[1], b[2].tolist())
        need = len(seq) - m
        if need > o.available_size():
            k = need + int(rng.integers(0, 64))
            assert o.evict(k)[0] == n.evict(k)
        if need <= o.available_size():
            s_o = o.alloc(need)
            assert s_o == n.alloc(need).tolist()
            assert o.insert(seq, list(slots) + s_o) == n.insert(seq, list(slots) + s_o)
        if step % 250 == 249:
            assert o.snapshot() == n.snapshot()
    assert o.snapshot() == n.snapshot()
    assert n.num_nodes() > 1000
