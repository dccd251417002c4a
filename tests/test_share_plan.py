"""Host plan of the shared-prefix decode (ra_decode_share_plan), on the CPU.

The plan must cover every request's positions 0 .. L-1 exactly once, and an
item may only group requests whose slot rows agree over its positions (then
reading the representative row once is the same as reading each member's).
Checked on a hand-traced batch and on random batches drawn from random radix
trees (shared runs, identical rows, rows that are prefixes of others, empty
contexts, permuted table rows, stride padding)."""
import numpy as np
import pytest

import paper_2312_07104_amd as pa


def check_plan(plan, rtt, rpi, lens, mpb, chunk):
    """Validity of a plan against its batch (independent of how it was built)."""
    B = len(lens)
    assert plan.batch == B and plan.members_per_item == mpb
    cover = [np.zeros(max(int(l), 0), dtype=np.int64) for l in lens]
    parts = [[] for _ in range(B)]
    prev_len = None
    rows = 0
    for row, t0, t1, moff, nm, *_ in plan.items:
        assert 0 <= t0 < t1 and t1 - t0 <= chunk
        assert 1 <= nm <= mpb
        if prev_len is not None:
            assert t1 - t0 <= prev_len  # longest first
        prev_len = t1 - t0
        rows += t1 - t0
        for b, p in plan.members[moff:moff + nm]:
            assert t1 <= lens[b]
            assert np.array_equal(rtt[rpi[b], t0:t1], rtt[row, t0:t1]), "member row differs over the item"
            cover[b][t0:t1] += 1
            parts[b].append(int(p))
    assert plan.rows_per_kv_head == rows
    assert plan.members.shape[0] == plan.n_member_entries
    n_parts = 0
    for b in range(B):
        assert np.all(cover[b] == 1), f"request {b}: positions not covered exactly once"
        lo, hi = int(plan.part_off[b]), int(plan.part_off[b + 1])
        if len(parts[b]) == 1:
            assert parts[b] == [-1] and hi == lo
        else:
            assert sorted(parts[b]) == list(range(lo, hi))
        n_parts += hi - lo
    assert plan.n_parts == n_parts == int(plan.part_off[B])
    return rows


def test_hand_traced_plan():
    """r0 = s + [20, 21], r1 = s + [30, 31, 32], r2 = r1 + [33, 34, 35], s =
    slots 1..10, r3 = [50, 51], r4 empty; min_shared 4, two members per item.
    Sorted r0 < r1 < r2 < r3 with neighbour common prefixes 10, 13, 0: s is
    shared by r0..r2 (blocks {r0, r1}, {r2}); the run 10..12 that r1 and r2
    also share is 3 < 4 positions, so it stays in their private parts."""
    s = list(range(1, 11))
    rows = [s + [20, 21], s + [30, 31, 32], s + [30, 31, 32, 33, 34, 35], [50, 51], []]
    stride = 20
    rtt = np.full((6, stride), -7, dtype=np.int32)  # padding past L never read
    rpi = np.array([4, 0, 2, 5, 1], dtype=np.int32)  # permuted table rows
    for b, r in enumerate(rows):
        rtt[rpi[b], :len(r)] = r
    lens = np.array([len(r) for r in rows], dtype=np.int32)
    plan = pa.ra_decode_share_plan(rtt, rpi, lens, members_per_item=2, min_shared=4, chunk_len=100)
    assert plan.chunk_len == 100
    want_items = [(rpi[0], 0, 10, [(0, 0), (1, 2)]), (rpi[0], 0, 10, [(2, 4)]), (rpi[2], 10, 16, [(2, 5)]),
                  (rpi[1], 10, 13, [(1, 3)]), (rpi[3], 0, 2, [(3, -1)]), (rpi[0], 10, 12, [(0, 1)])]
    assert plan.n_items == len(want_items)
    for (row, t0, t1, moff, nm, *_), (wr, w0, w1, wm) in zip(plan.items, want_items):
        assert (row, t0, t1) == (wr, w0, w1)
        assert [tuple(x) for x in plan.members[moff:moff + nm]] == wm
    assert list(plan.part_off) == [0, 2, 4, 6, 6, 6]
    assert check_plan(plan, rtt, rpi, lens, 2, 100) == 10 + 10 + 6 + 3 + 2 + 2


def random_batch(rng, n_req, depth, fanout, seg, private, dup_frac=0.1):
    """Requests on random root-to-node paths of a random tree of slot runs."""
    next_slot = [1000]

    def run(n):
        r = list(range(next_slot[0], next_slot[0] + n))
        next_slot[0] += n
        return r

    tree = {(): []}
    reqs = []
    for _ in range(n_req):
        path, toks = (), []
        for _ in range(int(rng.integers(0, depth + 1))):
            k = int(rng.integers(fanout))
            child = path + (k,)
            if child not in tree:
                tree[child] = run(int(rng.integers(seg[0], seg[1] + 1)))
            toks += tree[child]
            path = child
        if reqs and rng.random() < dup_frac:
            r = list(reqs[int(rng.integers(len(reqs)))])
            cut = int(rng.integers(0, len(r) + 1))
            toks = r[:cut]  # identical row or a prefix of another
        else:
            toks = toks[:int(rng.integers(0, len(toks) + 1))] if rng.random() < 0.2 else toks
            toks += run(int(rng.integers(0, private + 1)))
        reqs.append(toks)
    stride = max(1, max(len(t) for t in reqs) + 3)
    rpi = rng.permutation(n_req + 2)[:n_req].astype(np.int32)
    rtt = rng.integers(-5, 5, size=(n_req + 2, stride)).astype(np.int32)
    for b, t in enumerate(reqs):
        rtt[rpi[b], :len(t)] = t
    lens = np.array([len(t) for t in reqs], dtype=np.int32)
    return rtt, rpi, lens


@pytest.mark.parametrize("seed", range(12))
def test_random_plans_are_valid(seed):
    rng = np.random.default_rng(900 + seed)
    n_req = int(rng.integers(1, 120))
    rtt, rpi, lens = random_batch(rng, n_req, depth=4, fanout=3, seg=(1, 40), private=30)
    for mpb in (1, 3, 4, 16):
        for min_shared, chunk in ((1, 7), (8, 32), (32, 1000)):
            plan = pa.ra_decode_share_plan(rtt, rpi, lens, mpb, min_shared, chunk)
            rows = check_plan(plan, rtt, rpi, lens, mpb, chunk)
            assert rows <= int(lens.sum())


def test_shared_prefix_read_once_per_block():
    """All requests share a 500-position prefix: it is read once per block of
    members, and everything else once per request."""
    rng = np.random.default_rng(3)
    n, p = 37, 500
    rows = [list(range(p)) + list(range(10_000 + 100 * b, 10_000 + 100 * b + int(rng.integers(1, 90))))
            for b in range(n)]
    stride = max(len(r) for r in rows)
    rtt = np.zeros((n, stride), dtype=np.int32)
    for b, r in enumerate(rows):
        rtt[b, :len(r)] = r
    rpi = np.arange(n, dtype=np.int32)
    lens = np.array([len(r) for r in rows], dtype=np.int32)
    for mpb in (1, 4, 8):
        plan = pa.ra_decode_share_plan(rtt, rpi, lens, mpb, min_shared=64, chunk_len=128)
        rows_read = check_plan(plan, rtt, rpi, lens, mpb, 128)
        assert rows_read == -(-n // mpb) * p + int(lens.sum()) - n * p


def test_bad_arguments():
    rtt = np.zeros((2, 8), dtype=np.int32)
    with pytest.raises(pa.RadixAttnError):
        pa.ra_decode_share_plan(rtt, np.array([0, 2], np.int32), np.array([3, 3], np.int32), 2)  # row 2 > rows
    with pytest.raises(pa.RadixAttnError):
        pa.ra_decode_share_plan(rtt, np.array([0, 1], np.int32), np.array([3, 3], np.int32), 17)
    plan = pa.ra_decode_share_plan(rtt, np.zeros(0, np.int32), np.zeros(0, np.int32), 4)
    assert plan.n_items == 0 and list(plan.part_off) == [0]
