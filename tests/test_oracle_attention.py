"""Pins for the float64 attention oracle (CPU only).

The paper prints no numeric attention example, so the oracle is pinned by
what mathematics fixes: closed forms, brute-force scalar loops, an independent
library routine (torch's scaled-dot-product attention on the CPU in float64),
and invariants.  ``test_mutants_are_caught`` plants plausible mistakes in a
copy of the oracle and checks that some pin rejects every one of them.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import attention as oa
from workload import contentgen as cg
from workload import scenarios as S


def _rand(rng, *shape):
    return rng.standard_normal(shape)


# ---------------------------------------------------------------- pins ------
# Each pin takes the attention function under test so mutants can be fed in.

def pin_single_key(attend):
    rng = np.random.default_rng(1)
    q, k, v = _rand(rng, 1, 4, 8), _rand(rng, 1, 2, 8), _rand(rng, 1, 2, 8)
    out = attend(q, k, v, np.array([0]), 0.35)
    # one key: softmax weight exactly 1, the output is V itself
    for h in range(4):
        assert np.array_equal(out[0, h], v[0, h // 2])


def pin_zero_query_mean(attend):
    rng = np.random.default_rng(2)
    k, v = _rand(rng, 9, 1, 5), _rand(rng, 9, 1, 5)
    q = np.zeros((3, 2, 5))
    pos = np.array([2, 5, 8])
    out = attend(q, k, v, pos, 0.5)
    for r, p in enumerate(pos):
        np.testing.assert_allclose(out[r, 0], v[: p + 1, 0].mean(axis=0), rtol=0, atol=1e-14)
        np.testing.assert_allclose(out[r, 1], v[: p + 1, 0].mean(axis=0), rtol=0, atol=1e-14)


def pin_two_keys_logistic(attend):
    # D = 1: s_j = scale * q * k_j; weight of key 0 is the logistic 1/(1+e^(s1-s0)).
    q = np.array([[[1.5]]])
    k = np.array([[[2.0]], [[-0.5]]])
    v = np.array([[[3.0]], [[-7.0]]])
    scale = 0.8
    s0, s1 = scale * 1.5 * 2.0, scale * 1.5 * -0.5
    w0 = 1.0 / (1.0 + math.exp(s1 - s0))
    out = attend(q, k, v, np.array([1]), scale)
    assert abs(out[0, 0, 0] - (w0 * 3.0 + (1 - w0) * -7.0)) < 1e-13


def brute_force(q, k, v, q_pos, scale):
    """Scalar loops with math.exp; the group of head h is h // (Hq // Hkv)."""
    nq, hq, d = q.shape
    hkv = k.shape[1]
    grp = hq // hkv
    out = [[[0.0] * d for _ in range(hq)] for _ in range(nq)]
    for r in range(nq):
        for h in range(hq):
            g = h // grp
            scores = []
            for j in range(int(q_pos[r]) + 1):
                acc = 0.0
                for t in range(d):
                    acc += float(q[r, h, t]) * float(k[j, g, t])
                scores.append(scale * acc)
            mx = max(scores)
            w = [math.exp(s - mx) for s in scores]
            tot = sum(w)
            for t in range(d):
                out[r][h][t] = sum(w[j] * float(v[j, g, t]) for j in range(len(w))) / tot
    return np.array(out)


def pin_brute_force(attend):
    rng = np.random.default_rng(3)
    for hq, hkv, d, lk, nq in [(4, 2, 3, 7, 4), (6, 3, 2, 5, 5), (2, 2, 4, 6, 1), (8, 1, 3, 9, 3)]:
        q, k, v = _rand(rng, nq, hq, d), _rand(rng, lk, hkv, d), _rand(rng, lk, hkv, d)
        pos = np.sort(rng.choice(lk, size=nq, replace=False))
        np.testing.assert_allclose(attend(q, k, v, pos, 0.7), brute_force(q, k, v, pos, 0.7),
                                   rtol=0, atol=1e-12)


def pin_torch_sdpa(attend):
    """torch's causal SDPA (top-left aligned mask, grouped heads) over the full
    sequence; the last E rows are exactly the extend rows over a prefix P."""
    rng = np.random.default_rng(4)
    for hq, hkv, d, p, e in [(8, 2, 16, 13, 11), (4, 4, 8, 0, 9), (6, 1, 8, 20, 3)]:
        n = p + e
        q, k, v = _rand(rng, n, hq, d), _rand(rng, n, hkv, d), _rand(rng, n, hkv, d)
        scale = 1.0 / math.sqrt(d)
        ref = F.scaled_dot_product_attention(
            torch.from_numpy(q).permute(1, 0, 2)[None], torch.from_numpy(k).permute(1, 0, 2)[None],
            torch.from_numpy(v).permute(1, 0, 2)[None], is_causal=True, scale=scale,
            enable_gqa=True)[0].permute(1, 0, 2).numpy()
        out = attend(q[p:], k, v, np.arange(p, n), scale)
        np.testing.assert_allclose(out, ref[p:], rtol=0, atol=1e-12)


def pin_gqa_equals_repeated_mha(attend):
    rng = np.random.default_rng(5)
    hq, hkv, d, lk = 8, 2, 4, 6
    q, k, v = _rand(rng, 3, hq, d), _rand(rng, lk, hkv, d), _rand(rng, lk, hkv, d)
    pos = np.array([1, 3, 5])
    rep_k = np.repeat(k, hq // hkv, axis=1)
    rep_v = np.repeat(v, hq // hkv, axis=1)
    np.testing.assert_allclose(attend(q, k, v, pos, 0.4), attend(q, rep_k, rep_v, pos, 0.4), rtol=0, atol=1e-14)


def pin_decode_permutation_invariance(attend):
    rng = np.random.default_rng(6)
    q, k, v = _rand(rng, 1, 4, 6), _rand(rng, 10, 2, 6), _rand(rng, 10, 2, 6)
    perm = rng.permutation(10)
    a = attend(q, k, v, np.array([9]), 0.6)
    b = attend(q, k[perm], v[perm], np.array([9]), 0.6)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)


PINS = [pin_single_key, pin_zero_query_mean, pin_two_keys_logistic, pin_brute_force,
        pin_torch_sdpa, pin_gqa_equals_repeated_mha, pin_decode_permutation_invariance]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_oracle_pins(pin):
    pin(oa.attend)


# ---------------------------------------------------------- mutants ---------

def _mutant(kind):
    def attend(q, k, v, q_pos, scale):
        q = np.asarray(q, np.float64); k = np.asarray(k, np.float64); v = np.asarray(v, np.float64)
        nq, hq, d = q.shape
        hkv = k.shape[1]
        grp = hq // hkv
        out = np.zeros((nq, hq, d))
        for r in range(nq):
            last = int(q_pos[r]) + (0 if kind == "drop_own_key" else 1)
            if kind == "mask_one_extra":
                last = min(last + 1, k.shape[0])
            lo = 1 if kind == "drop_first_key" else 0
            for h in range(hq):
                g = (h % hkv) if kind == "gqa_modulo" else h // grp
                kk = k[lo:last, g, :]
                vv = v[lo:last, g, :]
                if kind == "transpose_kv":
                    kk, vv = vv, kk
                sc = -scale if kind == "sign" else scale
                s = sc * (kk @ q[r, h])
                if kind == "no_scale":
                    s = kk @ q[r, h]
                if len(s) == 0:
                    continue
                p = np.exp(s - s.max())
                if kind == "unnormalised":
                    out[r, h] = p @ vv
                else:
                    out[r, h] = (p / p.sum()) @ vv
        return out
    return attend


@pytest.mark.parametrize("kind", ["drop_own_key", "mask_one_extra", "drop_first_key", "gqa_modulo",
                                  "transpose_kv", "sign", "no_scale", "unnormalised"])
def test_mutants_are_caught(kind):
    """Every planted mistake fails at least one pin."""
    caught = []
    for pin in PINS:
        try:
            pin(_mutant(kind))
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"mutant {kind} passed every pin"


# ------------------------------------------- content-addressed requests -----

def test_extend_row_equals_decode_of_prefix():
    """Causal self-consistency: extend row i equals a decode over the first
    P+i+1 positions of the same sequence."""
    sc = S.cfg5_mixed_small()
    req = sc.phases[0].extend[0]
    p, e = req.prefix_len, req.extend_len
    rows = np.array([0, 1, e // 2, e - 1])
    ext = oa.extend_reference(req.tokens, p, e, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale, rows=rows)
    for r, i in enumerate(rows):
        dec = oa.decode_reference(req.tokens, p + i + 1, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale)
        np.testing.assert_allclose(ext[r], dec, rtol=0, atol=1e-14)


def test_reused_prefix_equals_recompute():
    """Two requests sharing a prefix see identical prefix keys and values, so a
    shared (cached) prefix and a private recomputation are the same input."""
    sc = S.cfg2_extend_fewshot(n_req=2, prefix_len=64, extend_len=8, heads=2, pool=1024)
    a, b = sc.phases[0].extend[0], sc.phases[0].extend[1]
    ka, va, _ = oa.request_kv(a.tokens, sc.seed, sc.hkv, sc.d)
    kb, vb, _ = oa.request_kv(b.tokens, sc.seed, sc.hkv, sc.d)
    assert np.array_equal(ka[:64], kb[:64]) and np.array_equal(va[:64], vb[:64])
    assert not np.array_equal(ka[64:], kb[64:])


def test_extend_rows_subset_matches_full():
    sc = S.cfg5_mixed_small()
    req = sc.phases[0].extend[1]
    full = oa.extend_reference(req.tokens, req.prefix_len, req.extend_len, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale)
    rows = np.array([3, 0, req.extend_len - 1])
    part = oa.extend_reference(req.tokens, req.prefix_len, req.extend_len, sc.seed, sc.hq, sc.hkv, sc.d,
                               sc.scale, rows=rows)
    np.testing.assert_allclose(part, full[rows], rtol=0, atol=1e-14)


def test_decode_single_token_context_returns_v():
    """L = 1: the decode output is the query token's own V, exactly."""
    toks = np.array([17], dtype=np.int32)
    out = oa.decode_reference(toks, 1, 99, 4, 2, 64, 0.125)
    h = cg.prefix_hashes(toks, 99)
    v = cg.values(h, cg.STREAM_V, 2, 64)[0]
    for hh in range(4):
        assert np.array_equal(out[hh], v[hh // 2].astype(np.float64))
