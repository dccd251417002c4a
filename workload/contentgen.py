"""Content-addressed synthetic values: the seeded inputs both sides share.

This module holds no attention and no radix-tree arithmetic.  It only turns
(seed, token sequence) into deterministic bf16 numbers, so that the oracle
and the GPU harness can each rebuild identical inputs on their own:

* ``prefix_hashes`` names every position of a token sequence by a 64-bit hash
  of the whole prefix up to and including it.  The paper notes that a token's
  KV cache depends only on the tokens before it (section 3, and Appendix A.1),
  so two requests that share a prefix share these hashes exactly.
* ``values_bf16`` maps (hash, stream, element) to an approximately standard
  normal bf16 value built from integers only (Irwin-Hall sum of twelve 16-bit
  uniforms), with no libm involved, so a HIP kernel can reproduce it bit for
  bit.

The random bits come from SplitMix64 (G. L. Steele, D. Lea, C. H. Flood,
"Fast splittable pseudorandom number generators", OOPSLA 2014), used as a
counter-based generator: output n of the stream that starts at state s is
mix(s + n * GAMMA).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_S30 = np.uint64(30)
_S27 = np.uint64(27)
_S31 = np.uint64(31)

# Stream identifiers folded into the per-token key.
STREAM_K = 1
STREAM_V = 2
STREAM_Q = 3
_STREAM_SALT = np.uint64(0xD1B54A32D192ED03)
_BASE_SALT = np.uint64(0x5851F42D4C957F2D)

# Irwin-Hall: twelve 16-bit uniforms x_k; z = (sum x_k - 393210) / 65536 has
# mean 0 and variance 12 * (65536^2 - 1) / (12 * 65536^2) ~= 1.
IH_TERMS = 12
IH_OFFSET = 393210  # 12 * 32767.5, the mean of the sum


def _u64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.uint64)


def mix64(z) -> np.ndarray:
    """SplitMix64 output function (the finaliser), elementwise, mod 2^64."""
    z = _u64(z)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> _S30)) * _M1
        z = (z ^ (z >> _S27)) * _M2
    return z ^ (z >> _S31)


def splitmix64_nth(state, n) -> np.ndarray:
    """Output number n (n >= 1) of SplitMix64 started at ``state``."""
    with np.errstate(over="ignore"):
        return mix64(_u64(state) + _u64(n) * GAMMA)


def base_hash(seed: int) -> np.uint64:
    """Hash of the empty prefix for a given seed."""
    return mix64(np.uint64(seed & 0xFFFFFFFFFFFFFFFF) ^ _BASE_SALT)[()]


def prefix_hashes_np(tokens: np.ndarray, seed: int) -> np.ndarray:
    """h[p] = mix((h[p-1] ^ t[p]) + GAMMA), h[-1] = base_hash(seed).

    Sequential along the sequence; returns uint64 [len(tokens)].
    """
    t = np.asarray(tokens, dtype=np.int64).astype(np.uint64)
    out = np.empty(t.shape[0], dtype=np.uint64)
    h = base_hash(seed)
    with np.errstate(over="ignore"):
        for p in range(t.shape[0]):
            h = mix64((h ^ t[p]) + GAMMA)[()]
            out[p] = h
    return out


def prefix_hashes_batch(seqs: list[np.ndarray], seed: int) -> list[np.ndarray]:
    """prefix_hashes for many sequences at once (vectorised across sequences)."""
    if not seqs:
        return []
    lens = np.array([len(s) for s in seqs], dtype=np.int64)
    n, lmax = len(seqs), int(lens.max()) if len(seqs) else 0
    tok = np.zeros((n, lmax), dtype=np.uint64)
    for i, s in enumerate(seqs):
        tok[i, : len(s)] = np.asarray(s, dtype=np.int64).astype(np.uint64)
    h = np.full(n, base_hash(seed), dtype=np.uint64)
    out = np.empty((n, lmax), dtype=np.uint64)
    with np.errstate(over="ignore"):
        for p in range(lmax):
            h = mix64((h ^ tok[:, p]) + GAMMA)
            out[:, p] = h
    return [out[i, : lens[i]].copy() for i in range(n)]


def token_key(hashes, stream: int) -> np.ndarray:
    """Per-(position, stream) SplitMix64 start state."""
    with np.errstate(over="ignore"):
        return mix64(_u64(hashes) ^ (np.uint64(stream) * _STREAM_SALT))


def f32_to_bf16_bits_rne(f: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round to nearest, ties to even) on the bits."""
    b = np.ascontiguousarray(f, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def values_bf16_bits_np(hashes, stream: int, n_elem: int) -> np.ndarray:
    """bf16 bit patterns, shape [len(hashes), n_elem].

    Element e of a position uses SplitMix64 outputs 3e+1, 3e+2, 3e+3 of the
    position's key; each 64-bit output gives four 16-bit uniforms.
    """
    key = token_key(np.atleast_1d(_u64(hashes)), stream)  # [P]
    out = np.empty((key.shape[0], n_elem), dtype=np.uint16)
    e = np.arange(n_elem, dtype=np.uint64)
    mask16 = np.uint64(0xFFFF)
    step = max(1, (1 << 22) // max(n_elem, 1))  # bound temporaries to ~4M elements
    for a in range(0, key.shape[0], step):
        kk = key[a : a + step, None]
        acc = np.zeros((kk.shape[0], n_elem), dtype=np.int64)
        for k in range(3):
            w = splitmix64_nth(kk, np.uint64(3) * e[None, :] + np.uint64(k + 1))
            for sh in (0, 16, 32, 48):
                acc += ((w >> np.uint64(sh)) & mask16).astype(np.int64)
        z = (acc - IH_OFFSET).astype(np.float32) * np.float32(1.0 / 65536.0)  # exact
        out[a : a + step] = f32_to_bf16_bits_rne(z)
    return out


# --- C fast path (same definitions; workload/csrc/contentgen.c) -------------

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcontentgen.so")
        if not os.path.exists(path):
            _LIB = False
        else:
            lib = ctypes.CDLL(path)
            lib.cg_prefix_hashes.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p]
            lib.cg_values_bf16.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]
            lib.cg_run_tokens.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p]
            _LIB = lib
    return _LIB or None


def prefix_hashes(tokens: np.ndarray, seed: int) -> np.ndarray:
    """Prefix hash chain (see prefix_hashes_np for the definition)."""
    lib = _lib()
    if lib is None:
        return prefix_hashes_np(tokens, seed)
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    out = np.empty(t.shape[0], dtype=np.uint64)
    lib.cg_prefix_hashes(t.ctypes.data, t.shape[0], seed & 0xFFFFFFFFFFFFFFFF, out.ctypes.data)
    return out


def values_bf16_bits(hashes, stream: int, n_elem: int) -> np.ndarray:
    """bf16 bit patterns [len(hashes), n_elem] (see values_bf16_bits_np)."""
    lib = _lib()
    if lib is None:
        return values_bf16_bits_np(hashes, stream, n_elem)
    h = np.ascontiguousarray(np.atleast_1d(_u64(hashes)))
    out = np.empty((h.shape[0], n_elem), dtype=np.uint16)
    lib.cg_values_bf16(h.ctypes.data, h.shape[0], stream, n_elem, out.ctypes.data)
    return out


def run_tokens_np(key: int, n: int, vocab: int) -> np.ndarray:
    """Token i of the synthetic text run named ``key``: mix(key + (i+1) GAMMA) mod vocab."""
    i = np.arange(1, n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return (mix64(np.uint64(key) + i * GAMMA) % np.uint64(vocab)).astype(np.int32)


def run_tokens(key: int, n: int, vocab: int) -> np.ndarray:
    lib = _lib()
    if lib is None:
        return run_tokens_np(key, n, vocab)
    out = np.empty(n, dtype=np.int32)
    lib.cg_run_tokens(int(key) & 0xFFFFFFFFFFFFFFFF, n, vocab, out.ctypes.data)
    return out


def values(hashes, stream: int, heads: int, dim: int, scale_pow2: int = 0) -> np.ndarray:
    """float32 array [P, heads, dim] holding exact bf16 values.

    ``scale_pow2`` multiplies by 2**scale_pow2 (exact in bf16), used to make
    sharper score distributions.
    """
    bits = values_bf16_bits(hashes, stream, heads * dim)
    v = bf16_bits_to_f32(bits).reshape(-1, heads, dim)
    if scale_pow2:
        v = v * np.float32(2.0 ** scale_pow2)
    return v
