"""Seeded workload recipes: token sequences and batch shapes for five workloads.

Each recipe yields a ``Scenario``:

* ``history``: finished requests replayed through the cache before the
  measured batch (they warm the cache, scatter slots and force evictions);
* ``phases``: batches of extend requests (cached prefix P, E new tokens) and
  decode requests (context of L tokens whose last token is new); after a phase
  its requests finish and their full sequences are inserted.

Token ids are uniform over a 32000-token vocabulary.  Shared text comes from a
lazily materialised random segment tree: a node is named by a 64-bit key, its
segment length is drawn from its key, and its tokens are
``contentgen.run_tokens(key)``.  Nothing here runs the radix tree or
attention; a scenario is plain data consumed by both sides.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable

import numpy as np

from . import contentgen as cg

VOCAB = 32000
SEED_BASE = 20231207


@dataclass
class ExtendReq:
    tokens: np.ndarray  # int32 [P + E]
    prefix_len: int
    extend_len: int


@dataclass
class DecodeReq:
    tokens: np.ndarray  # int32 [L]; the last token is the new query token
    seq_len: int


@dataclass
class Phase:
    extend: list[ExtendReq] = field(default_factory=list)
    decode: list[DecodeReq] = field(default_factory=list)


@dataclass
class Scenario:
    name: str
    seed: int
    hq: int
    hkv: int
    d: int
    pool_slots: int
    history_len: int
    history_fn: Callable[[int], np.ndarray]
    phases: list[Phase]
    q_scale_pow2: int = 0

    @property
    def scale(self) -> float:
        # 1/sqrt(D) as an fp32 number; both sides use exactly this value.
        return float(np.float32(1.0) / np.sqrt(np.float32(self.d)))

    def history(self, i: int) -> np.ndarray:
        return self.history_fn(i)

    def free_order(self) -> np.ndarray:
        """Initial FIFO order of free slots: a seeded permutation of [0, S)."""
        rng = np.random.default_rng(self.seed ^ 0x51A7)
        return rng.permutation(self.pool_slots).astype(np.int32)


def _key(*parts: int) -> int:
    h = np.uint64(0x243F6A8885A308D3)
    with np.errstate(over="ignore"):
        for p in parts:
            h = cg.mix64((h ^ np.uint64(p & 0xFFFFFFFFFFFFFFFF)) + cg.GAMMA)[()]
    return int(h)


class SegmentTree:
    """Infinite random tree of text segments, materialised on demand.

    Node keys: root children are _key(seed, 1, i); child j of node k is
    _key(k, 2, j).  Segment length of node k is lo + (mix(k) mod (hi-lo+1)).
    """

    def __init__(self, seed: int, branching: int, lo: int, hi: int):
        self.seed, self.b, self.lo, self.hi = seed, branching, lo, hi

    def child(self, key: int | None, j: int) -> int:
        return _key(self.seed, 1, j) if key is None else _key(key, 2, j)

    def seg_len(self, key: int) -> int:
        return self.lo + int(cg.mix64(np.uint64(key))[()] % np.uint64(self.hi - self.lo + 1))

    def tokens(self, key: int, n: int | None = None) -> np.ndarray:
        return cg.run_tokens(key, self.seg_len(key) if n is None else n, VOCAB)

    def random_path_tokens(self, rng: np.random.Generator, length: int) -> np.ndarray:
        """First ``length`` tokens of a random root-to-leaf walk (as deep as needed)."""
        parts, total, key = [], 0, None
        while total < length:
            key = self.child(key, int(rng.integers(self.b)))
            n = min(self.seg_len(key), length - total)
            parts.append(self.tokens(key, n))
            total += n
        return np.concatenate(parts) if parts else np.zeros(0, np.int32)


def _private(seed: int, tag: int, i: int, n: int) -> np.ndarray:
    return cg.run_tokens(_key(seed, 3, tag, i), n, VOCAB)


def _no_history(i: int) -> np.ndarray:
    raise IndexError(i)


# --------------------------------------------------------------------------
# The five workloads.  Sizes follow the recipe table of the design notes.
# --------------------------------------------------------------------------


def cfg1_decode_tiny(seed: int = SEED_BASE + 1) -> Scenario:
    """4 decode requests, MHA 8/8/64, one shared 128-token prefix plus private
    suffixes of U{16..64} tokens (the last being the query), pool 1024 slots."""
    rng = np.random.default_rng(seed)
    prefix = _private(seed, 0, 0, 128)
    reqs = []
    for r in range(4):
        s = int(rng.integers(16, 65))
        toks = np.concatenate([prefix, _private(seed, 1, r, s)])
        reqs.append(DecodeReq(toks, len(toks)))
    return Scenario("decode_tiny", seed, 8, 8, 64, 1024, 0, _no_history, [Phase(decode=reqs)])


def cfg2_extend_fewshot(seed: int = SEED_BASE + 2, n_req: int = 64, prefix_len: int = 2048,
                        extend_len: int = 128, heads: int = 32, pool: int = 262144) -> Scenario:
    """Few-shot: one cached shared prefix, each request extends private tokens.
    MHA 32/32/128, pool 262144 slots."""
    prefix = _private(seed, 0, 0, prefix_len)
    reqs = [ExtendReq(np.concatenate([prefix, _private(seed, 1, r, extend_len)]), prefix_len, extend_len)
            for r in range(n_req)]

    def hist(i: int) -> np.ndarray:
        if i != 0:
            raise IndexError(i)
        return prefix

    return Scenario("extend_fewshot", seed, heads, heads, 128, pool, 1, hist, [Phase(extend=reqs)])


def cfg3_decode_chat(seed: int = SEED_BASE + 3, n_req: int = 256, pool: int = 1048576) -> Scenario:
    """Multi-turn chat: a 4-ary tree with 3 levels below the root (84 edges of
    U[256, 1024] tokens); request r draws T ~ U[512, 4096] and a uniform leaf,
    takes the first min(T, path) tokens of the path and pads with private
    tokens to T.  GQA 32/8/128, pool 1048576 slots."""
    rng = np.random.default_rng(seed)
    tree = SegmentTree(seed, 4, 256, 1024)
    leaves = []
    for a in range(4):
        ka = tree.child(None, a)
        for b in range(4):
            kb = tree.child(ka, b)
            for c in range(4):
                leaves.append((ka, kb, tree.child(kb, c)))
    reqs = []
    for r in range(n_req):
        t = int(rng.integers(512, 4097))
        leaf = leaves[int(rng.integers(len(leaves)))]
        path = np.concatenate([tree.tokens(k) for k in leaf])
        toks = path[:t]
        if len(toks) < t:
            toks = np.concatenate([toks, _private(seed, 1, r, t - len(toks))])
        reqs.append(DecodeReq(toks, t))
    return Scenario("decode_chat", seed, 32, 8, 128, pool, 0, _no_history, [Phase(decode=reqs)])


def cfg4_branching(seed: int = SEED_BASE + 4, n_branch: int = 64, root_len: int = 8192,
                   branch_len: int = 512, extend_len: int = 64, pool: int = 262144) -> Scenario:
    """Tree-of-thought / self-consistency: an 8192-token root, 64 branches of
    512 private tokens; phase 1 extends 64 tokens per branch, phase 2 decodes
    one token per branch over all 8769 positions.  GQA 32/8/128."""
    root = _private(seed, 0, 0, root_len)
    ext, dec = [], []
    for b in range(n_branch):
        pre = np.concatenate([root, _private(seed, 1, b, branch_len)])
        toks = np.concatenate([pre, _private(seed, 2, b, extend_len)])
        ext.append(ExtendReq(toks, len(pre), extend_len))
        dtoks = np.concatenate([toks, _private(seed, 3, b, 1)])
        dec.append(DecodeReq(dtoks, len(dtoks)))
    return Scenario("branching", seed, 32, 8, 128, pool, 0, _no_history,
                    [Phase(extend=ext), Phase(decode=dec)])


def cfg5_mixed(seed: int = SEED_BASE + 5, n_ext: int = 32, n_dec: int = 512,
               n_history: int = 20000, pool: int = 4194304, branching: int = 4,
               ext_p=(1024, 8192), ext_e=(256, 2048), dec_l=(1024, 16384),
               hist_l=(256, 4096), hq: int = 64, hkv: int = 8) -> Scenario:
    """Continuous-batching mix, 70B-like GQA 64/8/128, pool 4194304 slots.

    A random segment tree (branching 4, segments U[256, 1024]) drives a
    history of 20000 finished requests (L ~ U[256, 4096], 100k tree calls),
    then one batch of 32 extend requests (P ~ U[1024, 8192] along a tree path,
    E ~ U[256, 2048] private) and 512 decode requests (L ~ U[1024, 16384]
    along tree paths).
    """
    rng = np.random.default_rng(seed)
    tree = SegmentTree(seed, branching, 256, 1024)
    ext, dec = [], []
    for r in range(n_ext):
        p = int(rng.integers(ext_p[0], ext_p[1] + 1))
        e = int(rng.integers(ext_e[0], ext_e[1] + 1))
        toks = np.concatenate([tree.random_path_tokens(rng, p), _private(seed, 1, r, e)])
        ext.append(ExtendReq(toks, p, e))
    for r in range(n_dec):
        l = int(rng.integers(dec_l[0], dec_l[1] + 1))
        toks = np.concatenate([tree.random_path_tokens(rng, l - 1), _private(seed, 2, r, 1)])
        dec.append(DecodeReq(toks, l))

    def hist(i: int) -> np.ndarray:
        if not 0 <= i < n_history:
            raise IndexError(i)
        hr = np.random.default_rng([seed, 7, i])
        l = int(hr.integers(hist_l[0], hist_l[1] + 1))
        priv = int(hr.integers(0, 65))
        return np.concatenate([tree.random_path_tokens(hr, max(l - priv, 1)), _private(seed, 4, i, priv)])

    return Scenario("mixed", seed, hq, hkv, 128, pool, n_history, hist, [Phase(extend=ext, decode=dec)])


def cfg5_mixed_small(seed: int = SEED_BASE + 5) -> Scenario:
    """Scaled-down mixed workload (same structure) small enough for the oracle."""
    sc = cfg5_mixed(seed, n_ext=4, n_dec=12, n_history=150, pool=24576, ext_p=(64, 700),
                    ext_e=(16, 200), dec_l=(64, 1500), hist_l=(32, 900), hq=16, hkv=2)
    sc.name = "mixed_small"
    return sc


def jump_forward(seed: int = SEED_BASE + 6, n_req: int = 256, ctx=(1024, 8192), ext=(2, 32),
                 hq: int = 32, hkv: int = 8, pool: int = 2097152) -> Scenario:
    """Jump-forward extends (the runtime effect of a compressed FSM, section 4):
    each request's context is a cached path of a random segment tree
    (L ~ U[ctx]), and it appends a deterministic run of E ~ U{ext} tokens in
    one extend instead of E decode steps.  GQA 32/8/128."""
    rng = np.random.default_rng(seed)
    tree = SegmentTree(seed, 4, 256, 1024)
    reqs = []
    for r in range(n_req):
        p = int(rng.integers(ctx[0], ctx[1] + 1))
        e = int(rng.integers(ext[0], ext[1] + 1))
        toks = np.concatenate([tree.random_path_tokens(rng, p), _private(seed, 1, r, e)])
        reqs.append(ExtendReq(toks, p, e))
    return Scenario("jump_forward", seed, hq, hkv, 128, pool, 0, _no_history, [Phase(extend=reqs)])


def jump_forward_small(seed: int = SEED_BASE + 6) -> Scenario:
    """Scaled-down jump-forward workload for full oracle comparison."""
    sc = jump_forward(seed, n_req=12, ctx=(40, 600), ext=(1, 33), pool=16384)
    sc.name = "jump_forward_small"
    return sc


def tp_shard(base: Callable[[], Scenario], hq: int, hkv: int, name: str) -> Callable[[], Scenario]:
    """One GPU's share of a tensor-parallel deployment: the same requests and
    slot tables with hq query heads and hkv kv heads (the head shard; the tree
    and slot ids are identical on every GPU)."""

    def make() -> Scenario:
        sc = base()
        sc.hq, sc.hkv, sc.name = hq, hkv, name
        return sc

    return make


ALL = {
    "decode_tiny": cfg1_decode_tiny,
    "extend_fewshot": cfg2_extend_fewshot,
    "decode_chat": cfg3_decode_chat,
    "branching": cfg4_branching,
    "mixed": cfg5_mixed,
    "mixed_small": cfg5_mixed_small,
    "jump_forward": jump_forward,
    "jump_forward_small": jump_forward_small,
    # tensor-parallel head shards: 32/8 heads at TP=4, 64/8 heads at TP=8
    "decode_chat_tp4": tp_shard(cfg3_decode_chat, 8, 2, "decode_chat_tp4"),
    "branching_tp4": tp_shard(cfg4_branching, 8, 2, "branching_tp4"),
    "mixed_tp8": tp_shard(cfg5_mixed, 8, 1, "mixed_tp8"),
}


def unique_context_tokens(sc: Scenario) -> int:
    """Distinct (prefix) positions over all final-batch sequences: an upper
    bound on the pool slots the final batch pins at once."""
    seen = set()
    total = 0
    for ph in sc.phases:
        seqs = [r.tokens for r in ph.extend] + [r.tokens for r in ph.decode]
        for h in cg.prefix_hashes_batch(seqs, sc.seed) if seqs else []:
            for x in h.tolist():
                if x not in seen:
                    seen.add(x)
                    total += 1
    return total
