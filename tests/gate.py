"""The parity gate and the needle keys that make it sensitive at long contexts.

Pure NumPy (no GPU): the CPU tests pin these helpers against planted mistakes
in oracle outputs, and the GPU tests use the same helpers on kernel outputs.

The gate is the spec bar for bf16 output against the float64 oracle
(max |err| <= 2e-2, mean |err| <= 2e-3) plus a relative-RMS bound of 1e-2.
With Q, K ~ N(0, 1) and scale 1/sqrt(D) the softmax is nearly flat: one
dropped or duplicated key moves a head's output by about 1/L per element,
about 1/sqrt(L) relative to the output itself.  At L = 2048 that breaks the
relative-RMS bound (0.017 to 0.027 for the mixed workload's head shape); at
L = 8769 and 16384 it gives about 0.008 and passes every bound.  Longer
contexts are therefore checked with needle keys: a planted key, set along one
query head's query, sized to take about half of that head's softmax mass.
Dropping it, counting it twice or reading a neighbour in its place then
moves that head's output by O(0.1 .. 0.5), far beyond the bounds.
"""
from __future__ import annotations

import numpy as np

MAX_ABS = 2e-2
MEAN_ABS = 2e-3
REL_RMS = 1e-2


def errors(got: np.ndarray, ref: np.ndarray) -> dict:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    e = np.abs(got - ref)
    return {"max": float(e.max()) if e.size else 0.0, "mean": float(e.mean()) if e.size else 0.0,
            "rel_rms": float(np.sqrt((e ** 2).sum() / max((ref ** 2).sum(), 1e-300)))}


def passes(er: dict) -> bool:
    return er["max"] <= MAX_ABS and er["mean"] <= MEAN_ABS and er["rel_rms"] <= REL_RMS


def assert_close(got, ref, what: str = "") -> dict:
    er = errors(got, ref)
    assert passes(er), f"{what}: {er}"
    return er


def to_bf16(x: np.ndarray) -> np.ndarray:
    """Round to bf16 (nearest, ties to even) and return the exact values as float32."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = ((b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)).astype(np.uint32)
    return (r << np.uint32(16)).view(np.float32)


def needle_key(q: np.ndarray, k_other: np.ndarray, scale: float, share: float = 0.5) -> np.ndarray:
    """A key row (bf16 values, float32 [D]) along query q that takes about
    ``share`` of the softmax mass of q over itself and the keys k_other
    [n, D]: its score s_n solves exp(s_n) = share / (1 - share) * sum_j
    exp(s_j).  The row is q times a scalar, rounded to bf16."""
    q64 = np.asarray(q, dtype=np.float64)
    s = float(scale) * (np.asarray(k_other, dtype=np.float64) @ q64) if len(k_other) else np.zeros(0)
    m = float(s.max()) if s.size else 0.0
    z = float(np.exp(s - m).sum()) if s.size else 1.0
    s_n = m + np.log(z * share / (1.0 - share))
    t = s_n / (float(scale) * float(q64 @ q64))
    return to_bf16((q64 * t).astype(np.float32))
