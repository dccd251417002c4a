"""GPU parity of extend attention with key splits (ra_extend_attention_split):
every item's keys cut into runs that separate work-groups process, partial
outputs merged by a second kernel.  Against the float64 oracle, with needle
keys on both sides of every split boundary, forced and library-picked split
counts, empty splits of short items, and the full-size head shard whose
work items alone would not fill the chip."""
import numpy as np
import pytest
import torch

from oracle import attention as oa
from workload import scenarios as S

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

import paper_2312_07104_amd as pa  # noqa: E402
from tests.harness import Needle, ScenarioRun, assert_close, errors, log, oracle_check, plant_needles  # noqa: E402
from tests.harness import make_scenario as _scenario  # noqa: E402

MIN_SPLIT_TILES = 8  # the kernel's smallest split (whole K/V tiles)


def _bf(t):
    return t.float().cpu().numpy()


def _shape(max_e, grp):
    """(query rows per work-group, keys per K/V tile) the launch takes."""
    return (256, 64) if max_e * grp >= 256 else (128, 32)


def split_starts(kend, bn, nsplit):
    """First key of each non-empty split of an item with kend keys."""
    nt = -(-kend // bn)
    ns = min(nsplit, max(1, nt // MIN_SPLIT_TILES))
    return [sp * nt // ns * bn for sp in range(ns)]


def _prep(sc):
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    torch.cuda.synchronize()
    return run, inp


def _check_rows(run, inp, out, what):
    sc = run.sc
    got = _bf(out)
    for toks, p, e, start in inp.ext_meta:
        if e == 0:
            continue
        ref = oa.extend_reference(toks, p, e, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale, sc.q_scale_pow2)
        assert_close(got[start:start + e], ref, f"{what} P={p} E={e}")


EXT = [(0, 1), (5, 130), (700, 63), (1500, 200), (63, 65), (2100, 7), (1, 0), (257, 129), (3000, 40)]


@pytest.mark.parametrize("num_splits", [0, 2, 3, 16])
@pytest.mark.parametrize("hq,hkv,d", [(8, 8, 64), (32, 8, 128), (8, 2, 128), (16, 1, 64)])
def test_split_extend_matches_oracle(hq, hkv, d, num_splits):
    """Both launch shapes (128 rows for G = 1 here, 256 rows otherwise), items
    from one tile to about fifty, so short items leave splits empty."""
    log(f"case: split extend hq={hq} hkv={hkv} d={d} num_splits={num_splits}")
    sc = _scenario("split", hq, hkv, d, 16384, extend=EXT, seed=200 + hq + d)
    run, inp = _prep(sc)
    ns = pa.ra_extend_num_splits(inp.n_ext, inp.max_extend_len, hq, hkv, num_splits)
    log(f"  splits per item: {ns}, workspace {run.extend_workspace_bytes(inp, num_splits)} bytes")
    assert ns == min(num_splits, 16) if num_splits else ns >= 1
    out = run.extend(inp, num_splits=num_splits)
    torch.cuda.synchronize()
    _check_rows(run, inp, out, f"split={num_splits}")


def test_one_split_is_the_plain_call():
    """num_splits = 1 launches exactly what ra_extend_attention launches."""
    log("case: one split equals the plain entry point")
    sc = _scenario("split1", 32, 8, 128, 16384, extend=EXT, seed=211)
    run, inp = _prep(sc)
    assert run.extend_workspace_bytes(inp, 1) == 0
    a = run.extend(inp)
    b = run.extend(inp, num_splits=1)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("hq,hkv,d,num_splits", [(32, 8, 128, 4), (8, 8, 64, 5), (16, 2, 128, 0)])
def test_split_boundary_needles(hq, hkv, d, num_splits):
    """A needle key (a key that takes a set share of the softmax) on each side
    of every split boundary, at the first and last keys, the last cached key,
    the first new key and the causal diagonal: a split that drops, repeats or
    misweights one key moves that row's output by about the needle's share."""
    ext = [(2500, 90), (1800, 33), (3100, 130)]
    log(f"case: split needles hq={hq} hkv={hkv} d={d} num_splits={num_splits}")
    sc = _scenario("split-needles", hq, hkv, d, 16384, extend=ext, seed=300 + hq + d)
    run, inp = _prep(sc)
    grp = hq // hkv
    rows_wg, bn = _shape(inp.max_extend_len, grp)
    tpb = rows_wg // grp
    ns = pa.ra_extend_num_splits(inp.n_ext, inp.max_extend_len, hq, hkv, num_splits)
    assert ns > 1
    needles, ext_rows = [], {}
    for r, (toks, P, E, start) in enumerate(inp.ext_meta):
        rows = sorted({0, E - 1, E // 2, min(E - 1, tpb), min(E - 1, tpb - 1)})
        ext_rows[r] = rows
        for k, i in enumerate(rows):
            tok_end = min(E, (i // tpb + 1) * tpb)  # end of the row's query tile
            starts = split_starts(P + tok_end, bn, ns)
            cands = [0, P - 1, P, P + i] + [s - 1 for s in starts[1:]] + starts[1:]
            cands = [c for c in cands if 0 <= c <= P + i]
            for j, pos in enumerate(cands):
                needles.append(Needle("ext", r, (r + 3 * k + 5 * j) % hq, pos, row=i, share=0.3))
    # one needle per (request, kv head, position): keep the first
    seen, uniq = set(), []
    for nd in needles:
        key = (nd.req, nd.head // grp, nd.pos)
        if key not in seen:
            seen.add(key)
            uniq.append(nd)
    log(f"  {len(uniq)} needles, splits per item {ns}")
    patches = plant_needles(run, inp, uniq)
    out = run.extend(inp, num_splits=num_splits)
    torch.cuda.synchronize()
    oracle_check(run, inp, out_ext=out, ext_rows=ext_rows, key_patches=patches, what="split needles")


def test_branching_tp4_split_sampled():
    """The head shard of the branching workload (8 / 2 heads, 64 extends of 64
    tokens over 8704 cached tokens): its 128 work items of 256 rows take one
    round of half the CUs, so the library splits their keys.  Needles at the
    split boundary of every sampled row's item, sampled rows against the
    oracle, and the split result against the unsplit call."""
    sc = S.ALL["branching_tp4"]()
    log(f"case: branching_tp4 split seed={sc.seed} Hq={sc.hq} Hkv={sc.hkv}")
    run, inp = _prep(sc)
    grp = sc.hq // sc.hkv
    ns = pa.ra_extend_num_splits(inp.n_ext, inp.max_extend_len, sc.hq, sc.hkv, 0)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    assert ns == min(16, -(-cus // (inp.n_ext * sc.hkv))) and ns > 1, ns
    plain = run.extend(inp)
    split = run.extend(inp, num_splits=0)
    torch.cuda.synchronize()
    er = errors(_bf(split), _bf(plain))
    log(f"  split vs unsplit {er}")
    assert er["max"] <= 2e-2
    rows_wg, bn = _shape(inp.max_extend_len, grp)
    needles, ext_rows = [], {}
    for r in (0, 17, 40, 63):
        toks, P, E, start = inp.ext_meta[r]
        starts = split_starts(P + E, bn, ns)
        ext_rows[r] = [0, 1, E // 2, E - 1]
        for k, i in enumerate(ext_rows[r]):
            for j, pos in enumerate([s - 1 for s in starts[1:]] + starts[1:] + [P - 1, P + i]):
                needles.append(Needle("ext", r, (2 * r + k + 3 * j) % sc.hq, pos, row=i, share=0.3))
    seen, uniq = set(), []
    for nd in needles:
        key = (nd.req, nd.head // grp, nd.pos)
        if key not in seen:
            seen.add(key)
            uniq.append(nd)
    patches = plant_needles(run, inp, uniq)
    out = run.extend(inp, num_splits=0)
    torch.cuda.synchronize()
    oracle_check(run, inp, out_ext=out, ext_rows=ext_rows, key_patches=patches, what="branching_tp4 split")


def test_split_arguments_rejected():
    sc = _scenario("split-args", 8, 2, 128, 4096, extend=[(100, 50), (30, 9)], seed=5)
    run, inp = _prep(sc)
    need = run.extend_workspace_bytes(inp, 4)
    assert need == 4 * inp.total_ext * sc.hq * (sc.d + 1) * 4
    with pytest.raises(pa.RadixAttnError):
        run.extend(inp, num_splits=-1)
    short = torch.empty(need - 16, dtype=torch.uint8, device="cuda")
    with pytest.raises(pa.RadixAttnError):
        run.extend(inp, num_splits=4, workspace=short)
    ok = torch.empty(need, dtype=torch.uint8, device="cuda")
    out = run.extend(inp, num_splits=4, workspace=ok)
    torch.cuda.synchronize()
    _check_rows(run, inp, out, "split=4 caller workspace")
