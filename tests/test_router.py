"""Data-parallel router (Appendix A.4): the native meta-tree against the
brute-force set model, the eviction log of the worker caches, the router's
view against the worker trees, and affinity dispatch against a single cache
of the same total size."""
import numpy as np
import pytest

import paper_2312_07104_amd as pa
from oracle.router import BruteRouter
from paper_2312_07104_amd.runtime import run_data_parallel


# ------------------------------------------------------- oracle pins -----

def test_oracle_router_hand_example():
    r = BruteRouter(2)
    r.insert(0, [1, 2, 3])
    r.insert(0, [1, 2, 4])
    r.insert(1, [1, 5])
    assert r.match([1, 2, 3, 9]) == [3, 1]
    assert r.match([1, 5, 5]) == [1, 2]
    assert r.held(0) == 4 and r.held(1) == 2  # (1) (1,2) (1,2,3) (1,2,4); (1) (1,5)
    # worker 0 drops the leaf [4] of path 1 2 4: only that position goes
    r.evict(0, [1, 2, 4], 1)
    assert r.match([1, 2, 4]) == [2, 1]
    assert r.match([1, 2, 3]) == [3, 1]
    # dropping the run 2 3 of path 1 2 3 takes everything through (1, 2)
    r.evict(0, [1, 2, 3], 2)
    assert r.match([1, 2, 3]) == [1, 1]
    assert r.held(0) == 1


def test_oracle_router_planted_mistake_fails_pin():
    class Off(BruteRouter):  # drops one position too few
        def evict(self, w, path, k):
            super().evict(w, path, k - 1)

    r = Off(1)
    r.insert(0, [1, 2, 4])
    r.evict(0, [1, 2, 4], 1)
    assert r.match([1, 2, 4]) != [2]


# ------------------------------------------- native router vs oracle -----

def _random_ops(seed, n_workers, n_ops, vocab=3, max_len=7):
    rng = np.random.default_rng(seed)
    nat, ref = pa.Router(n_workers), BruteRouter(n_workers)
    for _ in range(n_ops):
        w = int(rng.integers(n_workers))
        seq = rng.integers(0, vocab, size=int(rng.integers(1, max_len + 1))).astype(np.int32)
        if rng.random() < 0.6:
            nat.insert(w, seq)
            ref.insert(w, seq)
        else:
            k = int(rng.integers(0, len(seq) + 1))
            nat.evict(w, seq, k)
            ref.evict(w, seq, k)
        for _ in range(3):
            q = rng.integers(0, vocab, size=int(rng.integers(0, max_len + 2))).astype(np.int32)
            assert list(nat.match(q)) == ref.match(q), (q, nat.match(q), ref.match(q))
        assert [nat.held_tokens(x) for x in range(n_workers)] == [ref.held(x) for x in range(n_workers)]
    return nat


@pytest.mark.parametrize("seed,n_workers", [(1, 1), (2, 3), (3, 4), (4, 7)])
def test_native_router_matches_bruteforce(seed, n_workers):
    _random_ops(seed, n_workers, 400)


def test_native_router_frees_unheld_nodes():
    r = pa.Router(2)
    r.insert(0, [1, 2, 3, 4])
    r.insert(1, [1, 2, 9])
    assert r.num_nodes() == 4  # root, [1 2], [3 4], [9]
    r.evict(0, [1, 2, 3, 4], 2)
    r.evict(1, [1, 2, 9], 1)
    assert r.num_nodes() == 2  # root, [1 2] (still held by both)
    r.evict(0, [1, 2], 2)
    r.evict(1, [1, 2], 2)
    assert r.num_nodes() == 1 and r.held_tokens(0) == 0 and r.held_tokens(1) == 0


def test_data_parallel_argument_errors():
    seqs = _stream(13, 5)
    for kw in ({"commit_every": 0}, {"slack": -0.1}):
        with pytest.raises(ValueError):
            run_data_parallel(seqs, 2, 100, "affinity", **kw)
    with pytest.raises(ValueError):
        run_data_parallel(seqs, 2, 100, "best")


def test_router_argument_errors():
    with pytest.raises(pa.RadixAttnError):
        pa.Router(0)
    with pytest.raises(pa.RadixAttnError):
        pa.Router(65)
    r = pa.Router(2)
    with pytest.raises(pa.RadixAttnError):
        r.insert(2, [1])
    with pytest.raises(pa.RadixAttnError):
        r.evict(0, [1, 2], 3)


# ---------------------------------------------------- eviction log -----

def test_eviction_log_reports_freed_leaves():
    rng = np.random.default_rng(5)
    c = pa.RadixCache(64)
    c.log_evictions(True)
    inserted = []
    freed = 0
    for _ in range(60):
        seq = rng.integers(0, 4, size=int(rng.integers(1, 20))).astype(np.int32)
        node, m, slots = c.match_prefix(seq)
        need = len(seq) - m
        if need > c.available_size():
            freed += c.evict(need)
        if need <= c.available_size():
            c.insert(seq, np.concatenate([slots, c.alloc(need)]))
            inserted.append(tuple(seq.tolist()))
    logged = 0
    while True:
        e = c.pop_eviction()
        if e is None:
            break
        path, k = e
        assert 1 <= k <= len(path)
        assert any(s[: len(path)] == tuple(path.tolist()) for s in inserted)
        logged += k
    assert logged == freed > 0
    c.log_evictions(False)


# ------------------------------------------- router view vs workers -----

def _stream(seed, n_req, n_groups=6, prefix=40, suffix=(1, 30), vocab=50):
    rng = np.random.default_rng(seed)
    heads = [rng.integers(0, vocab, size=prefix).astype(np.int32) for _ in range(n_groups)]
    out = []
    for _ in range(n_req):
        g = int(rng.integers(n_groups))
        out.append(np.concatenate([heads[g], rng.integers(0, vocab, size=int(rng.integers(*suffix)))]).astype(np.int32))
    return out


@pytest.mark.parametrize("policy", ["affinity", "round_robin"])
def test_router_view_equals_worker_trees_with_immediate_commits(policy):
    seqs = _stream(11, 150)
    probes = seqs[::7] + [s[:20] for s in seqs[::11]]
    checks = []

    def probe(router, workers):
        for q in probes:
            m = router.match(q)
            for w, c in enumerate(workers):
                assert m[w] == c.match_prefix(q)[1]
        checks.append(1)

    res = run_data_parallel(seqs, 3, 160, policy, commit_every=1, probe=probe)
    assert len(checks) == len(seqs) + 1
    assert res.computed_tokens < res.prefill_tokens


def test_lazy_commits_keep_serving():
    seqs = _stream(12, 300)
    eager = run_data_parallel(seqs, 4, 200, "affinity", commit_every=1)
    lazy = run_data_parallel(seqs, 4, 200, "affinity", commit_every=40)
    assert lazy.prefill_tokens == eager.prefill_tokens
    assert abs(lazy.hit_rate - eager.hit_rate) < 0.1


# ---------------------------------------------- dispatch policies -----

def test_affinity_reaches_single_cache_hit_rate_and_balances():
    # Few-shot-like stream: 8 shared 300-token templates with short private
    # suffixes; each worker's cache fits about two templates, four workers
    # together fit all eight (a single cache of the same total size is the
    # best any dispatch can do).
    seqs = _stream(21, 800, n_groups=8, prefix=300, suffix=(5, 40), vocab=32000)
    per_worker = 2 * 300 + 400
    single = run_data_parallel(seqs, 1, 4 * per_worker, "least_loaded")
    res = {p: run_data_parallel(seqs, 4, per_worker, p, seed=3) for p in ("affinity", "round_robin", "random")}
    aff = res["affinity"]
    assert aff.hit_rate >= 0.95 * single.hit_rate
    assert aff.hit_rate > res["round_robin"].hit_rate + 0.1
    assert aff.hit_rate > res["random"].hit_rate + 0.1
    assert aff.imbalance < 1.5
