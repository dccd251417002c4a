"""GPU parity with needle keys where chunk, tile and diagonal mistakes sit.

At the lengths of the full-size workloads the plain gate cannot see one key
dropped, counted twice or read from a neighbouring position (see
``tests/test_parity_gate.py``).  Here needle keys (each takes about half of
one query head's softmax mass) are planted at the positions where such
mistakes would sit, on the launch shapes the workloads use: decode through
4096-, 2048- and 1024-token chunks (the first two in the longest-first item
order), the 256-row extend over an 8k prefix with 2k new tokens, the 128-row
extend of short runs over long prefixes, and both phases of the branching
workload (1024-token chunks, nine splits, needles in the shared root).
Every checked output is compared with the oracle, which sees the same
needles.
"""
import numpy as np
import pytest
import torch

from workload import scenarios as S

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only container
    pytest.skip("no GPU", allow_module_level=True)

import paper_2312_07104_amd as pa  # noqa: E402
from tests.harness import (Needle, ScenarioRun, check_table_pool, log, make_scenario, oracle_check,  # noqa: E402
                           plant_needles)


def _decode_lengths(rng, n):
    fixed = [16384, 16383, 16385 - 2, 12289, 12288, 12287, 8193, 8192, 8191, 4097, 4096, 4095, 2049, 2048, 2047,
             1025, 1024, 65, 33, 32, 1]
    return fixed + [int(x) for x in rng.integers(1, 16385, n - len(fixed))]


def _decode_needles(lens, hq, hkv, chunk):
    grp = hq // hkv
    needles = []
    for r, L in enumerate(lens):
        cands = sorted({p for p in (0, 1, 31, 32, 63, 64, chunk - 1, chunk, chunk + 1, 2 * chunk - 1, 2 * chunk,
                                    3 * chunk - 1, 3 * chunk, L // 2, L - 33, L - 32, L - 2, L - 1) if 0 <= p < L})
        for g in range(hkv):
            pos = cands[(r * hkv + g) % len(cands)]
            needles.append(Needle("dec", r, g * grp + (r + g) % grp, pos))
    return needles


@pytest.mark.parametrize("num_splits,q_pow2", [(4, 0), (4, 3), (8, 0), (16, 0)])
def test_decode_needles_long_contexts(num_splits, q_pow2):
    """40 decode requests up to 16384 tokens with the mixed workload's heads
    (64 / 8 / 128); chunks of 4096, 2048 and 1024 tokens; 320 needles at
    tile, chunk, middle and last positions; Q sharpened (x 8) in one case."""
    hq, hkv, d = 64, 8, 128
    lens = _decode_lengths(np.random.default_rng(90 + num_splits), 40)
    chunk = pa.ra_decode_chunk_len(len(lens), hkv, max(lens), num_splits)
    assert chunk == 16384 // num_splits
    log(f"case: decode needles chunk={chunk} q_pow2={q_pow2} requests={len(lens)}")
    sc = make_scenario(f"dneedle{num_splits}", hq, hkv, d, sum(lens) + 256, decode=lens, seed=91 + num_splits,
                       q_pow2=q_pow2)
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    torch.cuda.synchronize()
    patches = plant_needles(run, inp, _decode_needles(lens, hq, hkv, chunk))
    od = run.decode(inp, num_splits=num_splits)
    torch.cuda.synchronize()
    oracle_check(run, inp, out_dec=od, dec_reqs=range(len(lens)), key_patches=patches,
                 what=f"decode needles chunk={chunk}")


def _extend_needles(ext, hq, hkv, tile, rng):
    """(needles, rows to check per request) at the first and last cached
    key, the first new key, the causal diagonal and its neighbour, and tile
    edges of the prefix and of the new keys."""
    grp = hq // hkv
    needles, rows = [], {}
    for r, (P, E) in enumerate(ext):
        want = [(E - 1, 0), (0, max(P - 1, 0)), (0, P), (min(5, E - 1), P)]
        for i in (0, 1, tile - 1, tile, 2 * tile - 1, 2 * tile, E // 2, E - 1):
            if 0 <= i < E:
                want.append((i, P + i))          # the query's own key
                if P + i - 1 >= 0:
                    want.append((i, P + i - 1))  # the key just before it
        for pos in (tile - 1, tile, 2 * tile - 1, 2 * tile, P + tile - 1, P + tile):
            if 0 <= pos <= P + E - 1:
                want.append((E - 1, pos))
        seen = set()
        k = 0
        for i, pos in want:
            if (i, pos) in seen or pos > P + i:
                continue
            seen.add((i, pos))
            head = (r * 7 + k * 5) % hq  # spread the needles over kv heads
            needles.append(Needle("ext", r, head, pos, row=i))
            k += 1
        extra = rng.choice(E, min(E, 12), replace=False)
        rows[r] = sorted({i for i, _ in seen} | {0, E - 1} | set(int(x) for x in extra))
    return needles, rows


@pytest.mark.parametrize("shape", ["wide", "narrow"])
def test_extend_needles(shape):
    """wide: 64 / 8 / 128 heads, prefixes up to 8192 and up to 2048 new
    tokens (the 256-row kernel, 64-key tiles, longest-first items);
    narrow: 32 / 8 / 128 heads, 1 to 32 new tokens over prefixes up to 8192
    (the 128-row kernel, 32-key tiles).  Needles at the first and last cached
    key, the first new key, on the causal diagonal and next to it, and at tile
    edges; all needle rows and a sample of others against the oracle."""
    if shape == "wide":
        hq, hkv, tile = 64, 8, 64
        ext = [(8192, 2048), (8191, 2047), (8000, 1999), (0, 2048), (4096, 1024), (63, 65)]
    else:
        hq, hkv, tile = 32, 8, 32
        ext = [(8191, 32), (8192, 31), (4095, 2), (4096, 17), (1, 5), (0, 32), (3000, 1), (6000, 9)]
    d = 128
    rng = np.random.default_rng(7)
    log(f"case: extend needles {shape} {ext}")
    sc = make_scenario(f"eneedle_{shape}", hq, hkv, d, sum(p + e for p, e in ext) + 256, extend=ext, seed=97)
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    torch.cuda.synchronize()
    needles, rows = _extend_needles(ext, hq, hkv, tile, rng)
    patches = plant_needles(run, inp, needles)
    oe = run.extend(inp)
    torch.cuda.synchronize()
    oracle_check(run, inp, out_ext=oe, ext_rows=rows, key_patches=patches, what=f"extend needles {shape}")


def test_branching_needles_both_phases():
    """The branching workload as the bench runs it (32 / 8 / 128 heads):
    phase 1 extends 64 branches by 64 tokens over 8704 cached ones (needles
    in the shared root, at the branch start and on the diagonal), phase 2
    decodes all 64 branches over 8769 positions in 1024-token chunks (nine
    splits; needles at chunk edges of the shared root and in each branch).
    The table -> pool content check runs on both phases, all 64 requests of
    each phase against the oracle."""
    sc = S.cfg4_branching()
    grp = sc.hq // sc.hkv
    log(f"case: branching needles seed={sc.seed}")
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    torch.cuda.synchronize()
    log("table -> pool phase 1", check_table_pool(run, inp))
    P = inp.ext_meta[0][1]
    e_needles = []
    for r in range(inp.n_ext):
        for k, (i, pos) in enumerate([(0, P - 1), (0, P), (63, P + 63), (32, P + 31), (63, 0), (10, 8191),
                                      (10, 8192)]):
            if r % 4 == k % 4:
                e_needles.append(Needle("ext", r, (r + 3 * k) % sc.hq, pos, row=i))
    patches = plant_needles(run, inp, e_needles)
    oe = run.extend(inp)
    torch.cuda.synchronize()
    rows = {r: [0, 10, 31, 32, 63] for r in range(inp.n_ext)}
    oracle_check(run, inp, out_ext=oe, ext_rows=rows, key_patches=patches, what="branching extend needles")
    run.finish(0, inp)

    inp2 = run.prepare(1)
    run.store(inp2)
    torch.cuda.synchronize()
    log("table -> pool phase 2", check_table_pool(run, inp2, key_patches=patches))
    L = inp2.dec_meta[0][1]
    chunk = pa.ra_decode_chunk_len(inp2.n_dec, sc.hkv, inp2.max_seq_len, 0)
    assert chunk == 1024 and -(-L // chunk) == 9
    d_needles = []
    pos_list = [1023, 1024, 4095, 4096, 8191, 8192, 8703, 8704, 8767, 8768]
    for r in range(inp2.n_dec):
        for g in range(sc.hkv):
            if (r + g) % 3 == 0:
                pos = pos_list[(r + 5 * g) % len(pos_list)]
                d_needles.append(Needle("dec", r, g * grp + r % grp, pos))
    patches2 = plant_needles(run, inp2, d_needles, prior=patches)
    od = run.decode(inp2)
    torch.cuda.synchronize()
    oracle_check(run, inp2, out_dec=od, dec_reqs=range(inp2.n_dec), key_patches=patches2,
                 what="branching decode needles")
