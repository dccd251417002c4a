"""GPU parity of the shared-prefix decode (ra_decode_share_plan +
ra_decode_attention_shared) against the float64 oracle: batches on common
branches of the radix tree, every item boundary of sampled requests carrying a
needle key, member blocks of 1 .. 16 requests, the full-size chat, branching
and mixed decode batches."""
import numpy as np
import pytest
import torch

from oracle import attention as oa
from workload import contentgen as cg
from workload import scenarios as S

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

import paper_2312_07104_amd as pa  # noqa: E402
from tests.harness import Needle, ScenarioRun, assert_close, errors, log, oracle_check, plant_needles  # noqa: E402


def _bf(t):
    return t.float().cpu().numpy()


def tree_scenario(name, hq, hkv, d, seed, n_req=40, root=700, branch=(40, 300), n_branch=4, tail=(1, 200)):
    """Decode requests on a small radix tree: a shared root, a few branches,
    private tails; some requests stop inside the root, one repeats another's
    tokens exactly."""
    rng = np.random.default_rng(seed)
    rt = cg.run_tokens(seed * 7919, root, S.VOCAB)
    brs = [cg.run_tokens(seed * 7919 + 1 + k, int(rng.integers(*branch)), S.VOCAB) for k in range(n_branch)]
    dec = []
    for r in range(n_req):
        if rng.integers(4) == 0:
            toks = rt[: int(rng.integers(1, root + 1))]
        else:
            tl = cg.run_tokens(seed * 7919 + 100 + r, int(rng.integers(*tail)), S.VOCAB)
            toks = np.concatenate([rt, brs[int(rng.integers(n_branch))], tl])
        dec.append(S.DecodeReq(toks, len(toks)))
    dec.append(S.DecodeReq(dec[3].tokens.copy(), dec[3].seq_len))
    pool = sum(r.seq_len for r in dec) + 64
    return S.Scenario(name, seed, hq, hkv, d, pool, 0, lambda i: None, [S.Phase(decode=dec)])


def _prep(sc):
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    torch.cuda.synchronize()
    return run, inp


def _check_all(run, inp, out, what):
    sc = run.sc
    got = _bf(out)
    for i, (toks, l) in enumerate(inp.dec_meta):
        ref = oa.decode_reference(toks, l, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale, sc.q_scale_pow2)
        assert_close(got[i], ref, f"{what} decode req {i} L={l}")


@pytest.mark.parametrize("hq,hkv,d,mpb,min_shared,chunk", [
    (32, 8, 128, 4, 16, 1024), (32, 8, 128, 8, 64, 96), (32, 8, 128, 16, 256, 1024), (32, 8, 128, 1, 16, 64),
    (64, 8, 128, 2, 64, 1024), (64, 8, 128, 8, 16, 128), (8, 8, 64, 16, 64, 1024), (8, 8, 64, 3, 16, 40),
    (16, 1, 64, 1, 64, 1024), (16, 1, 64, 4, 16, 256), (6, 2, 64, 5, 32, 512), (12, 4, 128, 16, 32, 256)])
def test_shared_decode_matches_oracle(hq, hkv, d, mpb, min_shared, chunk):
    log(f"case: shared decode hq={hq} hkv={hkv} d={d} mpb={mpb} min_shared={min_shared} chunk={chunk}")
    sc = tree_scenario("tree", hq, hkv, d, seed=hq * 7 + d + mpb)
    run, inp = _prep(sc)
    plan, plan_dev = run.share_plan(inp, mpb, min_shared, chunk)
    lens = [l for _, l in inp.dec_meta]
    log(f"  items {plan.n_items} parts {plan.n_parts} rows {plan.rows_per_kv_head} of {sum(lens)}")
    assert plan.rows_per_kv_head < sum(lens) if mpb > 1 else plan.rows_per_kv_head == sum(lens)
    out = run.decode_shared(inp, plan, plan_dev)
    torch.cuda.synchronize()
    _check_all(run, inp, out, "shared")


def _boundary_needles(plan, inp, reqs, hq, grp):
    """A needle on each side of every item boundary of the given requests."""
    bounds = {b: set() for b in reqs}
    for row, t0, t1, moff, nm, *_ in plan.items:
        for b, _ in plan.members[moff:moff + nm]:
            if int(b) in bounds:
                bounds[int(b)].update({int(t0), int(t1) - 1})
    needles = []
    for b in reqs:
        L = inp.dec_meta[b][1]
        for k, pos in enumerate(sorted(bounds[b] | {0, L - 1})):
            if 0 <= pos < L:
                needles.append(Needle("dec", b, (b + 5 * k) % hq, pos, share=0.3))
    seen, uniq = set(), []
    for nd in needles:
        key = (nd.req, nd.head // grp, nd.pos)
        if key not in seen:
            seen.add(key)
            uniq.append(nd)
    return uniq


@pytest.mark.parametrize("mpb,chunk", [(4, 1024), (16, 200)])
def test_shared_decode_boundary_needles(mpb, chunk):
    """Needles at both ends of every item a sampled request takes part in: a
    shared run that drops, repeats or misweights a key at its edges moves
    the output by about the needle's share."""
    sc = tree_scenario("tree-needles", 32, 8, 128, seed=41, n_req=30, root=900)
    run, inp = _prep(sc)
    plan, plan_dev = run.share_plan(inp, mpb, 32, chunk)
    reqs = [0, 3, 7, 12, inp.n_dec - 1]
    needles = _boundary_needles(plan, inp, reqs, sc.hq, sc.hq // sc.hkv)
    log(f"  {len(needles)} needles over {plan.n_items} items")
    patches = plant_needles(run, inp, needles)
    out = run.decode_shared(inp, plan, plan_dev)
    torch.cuda.synchronize()
    oracle_check(run, inp, out_dec=out, dec_reqs=range(inp.n_dec), key_patches=patches, what="shared needles")


@pytest.mark.parametrize("mpb", [4, 8, 16])
def test_chat_shared_full(mpb):
    """The chat batch (256 requests on a 4-ary tree, 32 / 8 heads): every
    request against the oracle, with needles at the item boundaries of a
    sample, and against the per-request decode."""
    sc = S.cfg3_decode_chat()
    log(f"case: decode_chat shared mpb={mpb} seed={sc.seed}")
    run, inp = _prep(sc)
    plan, plan_dev = run.share_plan(inp, mpb)
    lens = [l for _, l in inp.dec_meta]
    log(f"  items {plan.n_items} parts {plan.n_parts} rows {plan.rows_per_kv_head} of {sum(lens)} "
        f"({plan.rows_per_kv_head / sum(lens):.3f}), plan {run.share_plan_seconds * 1e3:.1f} ms")
    ref = run.decode(inp)
    out = run.decode_shared(inp, plan, plan_dev)
    torch.cuda.synchronize()
    er = errors(_bf(out), _bf(ref))
    log(f"  shared vs per-request decode {er}")
    assert er["max"] <= 2e-2
    needles = _boundary_needles(plan, inp, [0, 17, 100, 255], sc.hq, sc.hq // sc.hkv)
    patches = plant_needles(run, inp, needles)
    out = run.decode_shared(inp, plan, plan_dev)
    torch.cuda.synchronize()
    oracle_check(run, inp, out_dec=out, dec_reqs=range(inp.n_dec), key_patches=patches, what="chat shared")


def test_branching_decode_shared_full():
    """64 branches over one 8192-token root: the root is read once per block
    of members; every request against the oracle."""
    sc = S.cfg4_branching()
    log(f"case: branching decode shared seed={sc.seed}")
    run = ScenarioRun(sc)
    inp0 = run.prepare(0)
    run.store(inp0)
    run.finish(0, inp0)
    inp = run.prepare(1)
    run.store(inp)
    torch.cuda.synchronize()
    plan, plan_dev = run.share_plan(inp)
    lens = [l for _, l in inp.dec_meta]
    log(f"  items {plan.n_items} parts {plan.n_parts} rows {plan.rows_per_kv_head} of {sum(lens)}")
    # the 8192-token root once per block of members, the rest once per request
    mpb = plan.members_per_item
    assert plan.rows_per_kv_head == -(-len(lens) // mpb) * 8192 + sum(l - 8192 for l in lens)
    needles = _boundary_needles(plan, inp, [0, 31, 63], sc.hq, sc.hq // sc.hkv)
    patches = plant_needles(run, inp, needles)
    out = run.decode_shared(inp, plan, plan_dev)
    torch.cuda.synchronize()
    oracle_check(run, inp, out_dec=out, dec_reqs=range(inp.n_dec), key_patches=patches, what="branching shared")


def test_mixed_decode_shared():
    """The headline batch's 512 decodes (64 / 8 heads, contexts up to 16k on
    a random segment tree): against the per-request decode for all, and the
    oracle for a sample."""
    sc = S.cfg5_mixed()
    log(f"case: mixed decode shared seed={sc.seed}")
    run, inp = _prep(sc)
    plan, plan_dev = run.share_plan(inp)
    lens = [l for _, l in inp.dec_meta]
    log(f"  items {plan.n_items} parts {plan.n_parts} rows {plan.rows_per_kv_head} of {sum(lens)}, "
        f"plan {run.share_plan_seconds * 1e3:.1f} ms")
    ref = run.decode(inp)
    out = run.decode_shared(inp, plan, plan_dev)
    torch.cuda.synchronize()
    er = errors(_bf(out), _bf(ref))
    log(f"  shared vs per-request decode {er}")
    assert er["max"] <= 2e-2
    lens = np.array(lens)
    sample = sorted({int(lens.argmax()), int(lens.argmin())} | set(range(0, inp.n_dec, 16)))
    oracle_check(run, inp, out_dec=out, dec_reqs=sample, what="mixed shared")


def test_shared_decode_arguments_rejected():
    sc = tree_scenario("tree-args", 8, 2, 128, seed=5, n_req=6)
    run, inp = _prep(sc)
    plan, plan_dev = run.share_plan(inp, 2, 16, 64)
    assert plan.n_parts > 0
    need = pa.ra_decode_shared_workspace_bytes(plan.n_parts, sc.hq, sc.d)
    with pytest.raises(pa.RadixAttnError):  # workspace too small
        run.decode_shared(inp, plan, plan_dev, workspace=torch.empty(need - 16, dtype=torch.uint8, device="cuda"))
    with pytest.raises(pa.RadixAttnError):  # plan words do not match the counts
        run.decode_shared(inp, plan, plan_dev[:-1])
    out = run.decode_shared(inp, plan, plan_dev, workspace=torch.empty(need, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    _check_all(run, inp, out, "caller workspace")


def test_mixed_shared_call_equals_separate_calls():
    """ra_mixed_attention_shared equals the extend call and the shared decode
    call bit for bit; a bad decode half fails the call before either half is
    queued (the extend output stays untouched)."""
    sc = S.cfg5_mixed_small()
    log(f"case: mixed shared call seed={sc.seed}")
    run, inp = _prep(sc)
    plan, plan_dev = run.share_plan(inp, min_shared=16)
    assert plan.n_parts > 0
    oe = run.extend(inp)
    od = run.decode_shared(inp, plan, plan_dev)
    me, md = run.mixed_shared(inp, plan, plan_dev)
    torch.cuda.synchronize()
    assert torch.equal(oe, me) and torch.equal(od, md)
    sentinel = torch.full_like(inp.q_ext, 7.0)
    with pytest.raises(pa.RadixAttnError):
        pa.ra_mixed_attention_shared(
            inp.q_ext, inp.k_new[: inp.total_ext], inp.v_new[: inp.total_ext], inp.rpi[: inp.n_ext],
            inp.prefix_lens, inp.extend_lens, inp.extend_start, inp.max_extend_len, inp.q_dec, plan, plan_dev[:-1],
            run.k_pool, run.v_pool, inp.table, sc.scale, out_ext=sentinel)
    torch.cuda.synchronize()
    assert bool((sentinel == 7.0).all())


def test_mixed_shared_call_with_an_empty_half():
    """ra_mixed_attention_shared with no extend tokens runs only the shared
    decode, and with no decode requests (the plan of an empty batch) only the
    extend: outputs equal the single calls bit for bit."""
    sc = S.cfg5_mixed_small()
    log(f"case: mixed shared call with an empty half seed={sc.seed}")
    run, inp = _prep(sc)
    plan, plan_dev = run.share_plan(inp, min_shared=16)
    od = run.decode_shared(inp, plan, plan_dev)
    oe = run.extend(inp)
    z = torch.zeros(0, dtype=torch.int32, device="cuda")
    _, md = pa.ra_mixed_attention_shared(
        inp.q_ext[:0], inp.k_new[:0], inp.v_new[:0], z, z, z, z, 0, inp.q_dec, plan, plan_dev,
        run.k_pool, run.v_pool, inp.table, sc.scale)
    eplan = pa.ra_decode_share_plan(inp.table_host, np.zeros(0, np.int32), np.zeros(0, np.int32), 4)
    assert eplan.n_items == 0
    eplan_dev = torch.from_numpy(eplan.words).to("cuda")
    me, _ = pa.ra_mixed_attention_shared(
        inp.q_ext, inp.k_new[: inp.total_ext], inp.v_new[: inp.total_ext], inp.rpi[: inp.n_ext], inp.prefix_lens,
        inp.extend_lens, inp.extend_start, inp.max_extend_len, inp.q_dec[:0], eplan, eplan_dev,
        run.k_pool, run.v_pool, inp.table, sc.scale)
    torch.cuda.synchronize()
    assert torch.equal(md, od) and torch.equal(me, oe)
