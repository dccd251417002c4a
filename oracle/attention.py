"""Float64 causal softmax attention, recomputed per request with no cache.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Definition (the textbook attention the paper builds on, section 3; a token's
keys and values depend only on the tokens before it, section 3 and Appendix
A.1, so reusing a cached prefix must give exactly this result).  For a query
at position i with query head h and key/value head g = floor(h / G), where
G = Hq / Hkv (query heads are grouped contiguously onto key/value heads):

    s_j = scale * sum_d Q[i, h, d] * K[j, g, d]      for j = 0 .. i
    p_j = exp(s_j - max_k s_k) / sum_k exp(s_k - max_k s_k)
    O[i, h, :] = sum_j p_j * V[j, g, :]

Extend (prefill of new tokens over a cached prefix, Appendix A.1): queries are
the new positions P .. P+E-1.  Decode: one query at position L-1 over keys
0 .. L-1, including its own.

Parity is pinned by closed forms, brute-force scalar loops, a library routine
(torch's scaled-dot-product attention in float64 on the CPU) and invariants;
the paper prints no numeric attention example, so no value here is pinned to a
printed number.
"""
from __future__ import annotations

import time

import numpy as np

from workload import contentgen as cg


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: np.ndarray, scale: float) -> np.ndarray:
    """Causal attention for one request.

    q: [nq, Hq, D]; k, v: [Lk, Hkv, D]; q_pos: [nq] absolute positions (query
    r sees keys 0 .. q_pos[r]).  Returns float64 [nq, Hq, D].
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    q_pos = np.asarray(q_pos, dtype=np.int64)
    nq, hq, d = q.shape
    lk, hkv, _ = k.shape
    if hq % hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    if nq and (q_pos.max() >= lk or q_pos.min() < 0):
        raise ValueError("query position outside the key range")
    grp = hq // hkv
    n_keys = int(q_pos.max()) + 1 if nq else 0
    out = np.zeros((nq, hq, d), dtype=np.float64)
    if nq == 0:
        return out
    allowed = np.arange(n_keys)[None, :] <= q_pos[:, None]  # [nq, n_keys]
    for h in range(hq):
        g = h // grp
        s = float(scale) * (q[:, h, :] @ k[:n_keys, g, :].T)  # [nq, n_keys]
        s = np.where(allowed, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        p = np.exp(s - m)
        p /= p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:n_keys, g, :]
    return out


def request_kv(tokens: np.ndarray, seed: int, hkv: int, d: int, upto: int | None = None,
               key_patches: dict | None = None):
    """Regenerate a request's K and V [L, Hkv, D] from its own token list.

    ``key_patches`` overrides inputs: {prefix hash: {kv head: K row [D]}}.  A
    position whose prefix hash is listed takes that K row for that kv head
    (a test plants such keys in the pool, so every request whose context
    holds the same prefix sees the same key, as the pool would serve it).
    """
    t = np.asarray(tokens)[: len(tokens) if upto is None else upto]
    h = cg.prefix_hashes(t, seed)
    k = cg.values(h, cg.STREAM_K, hkv, d)
    if key_patches:
        for p in np.flatnonzero(np.isin(h, np.fromiter(key_patches.keys(), dtype=np.uint64))):
            for g, row in key_patches[int(h[p])].items():
                k[p, g] = row
    return k, cg.values(h, cg.STREAM_V, hkv, d), h


def extend_reference(tokens: np.ndarray, prefix_len: int, extend_len: int, seed: int,
                     hq: int, hkv: int, d: int, scale: float, q_scale_pow2: int = 0,
                     rows: np.ndarray | None = None, key_patches: dict | None = None,
                     timings: dict | None = None) -> np.ndarray:
    """Output rows of an extend request, float64 [len(rows) or E, Hq, D].

    ``rows`` selects new-token indices (0 .. E-1) to compute; default all.
    ``key_patches`` as in ``request_kv``.  ``timings``, when given, gets the
    seconds spent regenerating inputs ("regen") and attending ("attend").
    """
    t0 = time.perf_counter()
    n = prefix_len + extend_len
    k, v, h = request_kv(tokens, seed, hkv, d, upto=n, key_patches=key_patches)
    rows = np.arange(extend_len) if rows is None else np.asarray(rows, dtype=np.int64)
    q = cg.values(h[prefix_len + rows], cg.STREAM_Q, hq, d, q_scale_pow2)
    t1 = time.perf_counter()
    out = attend(q, k, v, prefix_len + rows, scale)
    if timings is not None:
        timings["regen"] = timings.get("regen", 0.0) + t1 - t0
        timings["attend"] = timings.get("attend", 0.0) + time.perf_counter() - t1
    return out


def decode_reference(tokens: np.ndarray, seq_len: int, seed: int, hq: int, hkv: int, d: int,
                     scale: float, q_scale_pow2: int = 0, key_patches: dict | None = None,
                     timings: dict | None = None) -> np.ndarray:
    """Output of a decode request (query at position L-1), float64 [Hq, D].
    ``key_patches`` and ``timings`` as in ``extend_reference``."""
    t0 = time.perf_counter()
    k, v, h = request_kv(tokens, seed, hkv, d, upto=seq_len, key_patches=key_patches)
    q = cg.values(h[seq_len - 1 : seq_len], cg.STREAM_Q, hq, d, q_scale_pow2)
    t1 = time.perf_counter()
    out = attend(q, k, v, np.array([seq_len - 1]), scale)[0]
    if timings is not None:
        timings["regen"] = timings.get("regen", 0.0) + t1 - t0
        timings["attend"] = timings.get("attend", 0.0) + time.perf_counter() - t1
    return out
