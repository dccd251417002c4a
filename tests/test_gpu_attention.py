"""GPU parity: the HIP path (through the C ABI) against the float64 oracle.

Every case prints its name, seed and shapes before touching the GPU.  Full-size
workloads are compared on sampled requests / rows the oracle recomputes one by
one; the small ones in full.
"""
import numpy as np
import pytest
import torch

from oracle import attention as oa
from workload import contentgen as cg
from workload import scenarios as S

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only container
    pytest.skip("no GPU", allow_module_level=True)

import paper_2312_07104_amd as pa  # noqa: E402
from tests.harness import (Needle, ScenarioRun, assert_close, check_table_pool, errors, log,  # noqa: E402
                           oracle_check, plant_needles)


def _bf(t):
    return t.float().cpu().numpy()


def run_phase(run, idx, num_splits=0):
    inp = run.prepare(idx)
    run.store(inp)
    oe = run.extend(inp)
    od = run.decode(inp, num_splits=num_splits)
    torch.cuda.synchronize()
    return inp, oe, od


def check_decode(run, inp, od, sample=None, what=""):
    sc = run.sc
    idx = range(inp.n_dec) if sample is None else sample
    got = _bf(od)
    worst = None
    for i in idx:
        toks, L = inp.dec_meta[i]
        ref = oa.decode_reference(toks, L, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale, sc.q_scale_pow2)
        er = assert_close(got[i], ref, f"{what} decode req {i} L={L}")
        worst = er if worst is None or er["max"] > worst["max"] else worst
    return worst


def check_extend(run, inp, oe, sample=None, rows_per_req=None, what="", seed=0):
    sc = run.sc
    rng = np.random.default_rng(seed)
    idx = range(inp.n_ext) if sample is None else sample
    got = _bf(oe)
    worst = None
    for i in idx:
        toks, p, e, start = inp.ext_meta[i]
        rows = np.arange(e) if rows_per_req is None or rows_per_req >= e else np.unique(
            np.concatenate([[0, e - 1], rng.choice(e, rows_per_req, replace=False)]))
        ref = oa.extend_reference(toks, p, e, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale, sc.q_scale_pow2, rows=rows)
        er = assert_close(got[start + rows], ref, f"{what} extend req {i} P={p} E={e}")
        worst = er if worst is None or er["max"] > worst["max"] else worst
    return worst


# ----------------------------------------------------------- generator -----

def test_gpu_generator_bit_exact():
    log("case: generator bit-exact, 3000 positions x 1024")
    h = cg.prefix_hashes(np.arange(3000, dtype=np.int32) % 977, 11)
    out = torch.empty((3000, 8, 128), dtype=torch.bfloat16, device="cuda")
    from workload import gpu_gen
    gpu_gen.fill(out, h, cg.STREAM_V)
    got = out.view(torch.int16).cpu().numpy().view(np.uint16).reshape(3000, -1)
    assert np.array_equal(got, cg.values_bf16_bits(h, cg.STREAM_V, 1024))
    rows = np.random.default_rng(0).permutation(3000)[:500]
    out2 = torch.zeros((3000, 8, 128), dtype=torch.bfloat16, device="cuda")
    gpu_gen.fill(out2, h[:500], cg.STREAM_K, rows=rows, scale_pow2=2)
    got2 = out2.float().cpu().numpy()[rows]
    assert np.array_equal(got2, cg.values(h[:500], cg.STREAM_K, 8, 128, 2))


# ------------------------------------------------------------ store_kv -----

@pytest.mark.parametrize("hkv,d", [(8, 64), (8, 128), (2, 128)])
def test_store_kv_bit_exact(hkv, d):
    import paper_2312_07104_amd as pa
    log(f"case: store_kv hkv={hkv} d={d}")
    rng = np.random.default_rng(hkv * d)
    S_ = 5000
    n = 777
    slots = rng.choice(S_, n, replace=False).astype(np.int32)
    slots[5] = -1          # skipped
    slots[9] = S_ + 3      # skipped
    kp = torch.zeros((S_, hkv, d), dtype=torch.bfloat16, device="cuda")
    vp = torch.zeros_like(kp)
    kn = torch.randn((n, hkv, d), device="cuda").bfloat16()
    vn = torch.randn((n, hkv, d), device="cuda").bfloat16()
    pa.ra_store_kv(torch.from_numpy(slots).cuda(), kn, vn, kp, vp)
    torch.cuda.synchronize()
    ok = (slots >= 0) & (slots < S_)
    s = torch.from_numpy(slots[ok]).long().cuda()
    assert torch.equal(kp[s], kn[torch.from_numpy(ok).cuda()])
    assert torch.equal(vp[s], vn[torch.from_numpy(ok).cuda()])
    untouched = np.ones(S_, bool)
    untouched[slots[ok]] = False
    assert int(kp[torch.from_numpy(untouched).cuda()].abs().sum()) == 0


# --------------------------------------------------------- full configs -----

def test_decode_tiny_full():
    sc = S.cfg1_decode_tiny()
    log(f"case: decode_tiny seed={sc.seed}")
    run = ScenarioRun(sc)
    inp, _, od = run_phase(run, 0)
    er = check_decode(run, inp, od, what="decode_tiny")
    log("decode_tiny worst", er)


@pytest.fixture(scope="module")
def fewshot():
    sc = S.cfg2_extend_fewshot()
    log(f"case: extend_fewshot seed={sc.seed}")
    run = ScenarioRun(sc)
    inp, oe, _ = run_phase(run, 0)
    return run, inp, oe


def test_extend_fewshot_sampled(fewshot):
    run, inp, oe = fewshot
    er = check_extend(run, inp, oe, sample=[0, 17, 63], what="extend_fewshot")
    log("extend_fewshot worst", er)


@pytest.fixture(scope="module")
def chat():
    sc = S.cfg3_decode_chat()
    log(f"case: decode_chat seed={sc.seed}")
    run = ScenarioRun(sc)
    inp, _, od = run_phase(run, 0)
    return run, inp, od


def test_decode_chat_sampled(chat):
    run, inp, od = chat
    lens = np.array([l for _, l in inp.dec_meta])
    sample = sorted({int(lens.argmin()), int(lens.argmax()), 0, 100, 255})
    er = check_decode(run, inp, od, sample=sample, what="decode_chat")
    log("decode_chat worst", er)


def test_decode_splits_agree(chat):
    run, inp, od = chat
    sample = [3, 77]
    for ns in (1, 2, 7):
        log(f"case: decode_chat num_splits={ns}")
        o2 = run.decode(inp, num_splits=ns)
        torch.cuda.synchronize()
        check_decode(run, inp, o2, sample=sample, what=f"splits={ns}")
        assert errors(_bf(o2), _bf(od))["max"] <= 2e-2


def test_branching_two_phases():
    sc = S.cfg4_branching()
    log(f"case: branching seed={sc.seed}")
    run = ScenarioRun(sc)
    inp, oe, _ = run_phase(run, 0)
    er = check_extend(run, inp, oe, sample=[0, 31, 63], rows_per_req=24, what="branching/extend")
    log("branching extend worst", er)
    run.finish(0, inp)
    inp2, _, od = run_phase(run, 1)
    # decode contexts hit the pool written by store_kv in phase 1
    assert all(m == c for m, c in zip(inp2.plan.matched, inp2.plan.ctx_lens))
    er = check_decode(run, inp2, od, sample=[0, 1, 40, 63], what="branching/decode")
    log("branching decode worst", er)


def test_mixed_full_size():
    """The headline batch (64 / 8 / 128 heads, 32 extends and 512 decodes over
    a 4,194,304-slot pool) through the one mixed call, as bench.py launches
    it.  The table -> pool content check covers every attended position; the
    mixed call equals separate calls bit for bit; then needles go to the
    decode chunk edges (4096-token chunks, longest-first order), the first
    and last positions, and to the extends' last cached key, first new key,
    causal diagonal and tile edges.  Every decode request and every extend
    request (needle rows plus a sample of others) against the oracle."""
    sc = S.cfg5_mixed()
    grp = sc.hq // sc.hkv
    log(f"case: mixed seed={sc.seed} (history replay on host)")
    run = ScenarioRun(sc)
    log(f"history ops={run.history_ops} in {run.history_seconds:.2f}s")
    inp, oe_sep, od_sep = run_phase(run, 0)
    oe, od = run.mixed(inp)
    torch.cuda.synchronize()
    assert torch.equal(oe, oe_sep) and torch.equal(od, od_sep)
    log("table -> pool", check_table_pool(run, inp))
    chunk = pa.ra_decode_chunk_len(inp.n_dec, sc.hkv, inp.max_seq_len, 0)
    assert chunk == 4096
    needles = []
    lens = [l for _, l in inp.dec_meta]
    long_reqs = [r for r, l in enumerate(lens) if l > 3 * chunk][:24]
    for r in long_reqs:
        L = lens[r]
        cands = [0, 31, 32, chunk - 1, chunk, 2 * chunk - 1, 2 * chunk, 3 * chunk - 1, 3 * chunk, L - 2, L - 1]
        for g in range(sc.hkv):
            needles.append(Needle("dec", r, g * grp + (r + g) % grp, cands[(r + 3 * g) % len(cands)]))
    rng = np.random.default_rng(55)
    ext_rows = {}
    for r, (toks, P, E, start) in enumerate(inp.ext_meta):
        want = [(0, P - 1), (0, P), (E - 1, 0), (63, P + 63), (64, P + 64), (64, P + 63), (E - 1, P + E - 1),
                (E - 1, 64), (E - 1, P + 64)]
        for k, (i, pos) in enumerate(want):
            if (r + k) % 3 == 0 and i < E and pos <= P + i:
                needles.append(Needle("ext", r, (5 * r + 11 * k) % sc.hq, pos, row=i))
        ext_rows[r] = sorted({0, 63, 64, E - 1} | {i for i, _ in want if i < E} |
                             set(int(x) for x in rng.choice(E, 6, replace=False)))
    log(f"planting {len(needles)} needles")
    patches = plant_needles(run, inp, needles)
    oe, od = run.mixed(inp)
    torch.cuda.synchronize()
    oracle_check(run, inp, out_ext=oe, out_dec=od, ext_rows=ext_rows, dec_reqs=range(inp.n_dec),
                 key_patches=patches, what="mixed full size")


def test_mixed_small_full():
    sc = S.cfg5_mixed_small()
    log(f"case: mixed_small seed={sc.seed}")
    run = ScenarioRun(sc)
    inp, oe, od = run_phase(run, 0)
    check_extend(run, inp, oe, what="mixed_small/extend")
    check_decode(run, inp, od, what="mixed_small/decode")


# ------------------------------------------- jump-forward (small-E) extends -----

def test_jump_forward_small_full():
    sc = S.jump_forward_small()
    log(f"case: jump_forward_small seed={sc.seed}")
    run = ScenarioRun(sc)
    inp, oe, _ = run_phase(run, 0)
    assert max(e for _, _, e, _ in inp.ext_meta) <= 33
    er = check_extend(run, inp, oe, what="jump_forward_small")
    log("jump_forward_small worst", er)


def test_jump_forward_sampled():
    sc = S.jump_forward()
    log(f"case: jump_forward seed={sc.seed}")
    run = ScenarioRun(sc)
    inp, oe, _ = run_phase(run, 0)
    lens = np.array([e for _, _, e, _ in inp.ext_meta])
    sample = sorted({int(lens.argmin()), int(lens.argmax()), 0, 101, 255})
    er = check_extend(run, inp, oe, sample=sample, what="jump_forward")
    log("jump_forward worst", er)


# ----------------------------------------------- tensor-parallel head shards -----

def test_tp8_mixed_shard_sampled():
    sc = S.ALL["mixed_tp8"]()
    log(f"case: mixed_tp8 seed={sc.seed} Hq={sc.hq} Hkv={sc.hkv}")
    run = ScenarioRun(sc)
    inp, oe, od = run_phase(run, 0)
    me, md = run.mixed(inp)  # one kv head, G = 8
    torch.cuda.synchronize()
    assert torch.equal(me, oe) and torch.equal(md, od)
    check_extend(run, inp, oe, sample=[1, 30], rows_per_req=12, what="mixed_tp8/extend")
    lens = np.array([l for _, l in inp.dec_meta])
    check_decode(run, inp, od, sample=sorted({int(lens.argmax()), int(lens.argmin()), 77}), what="mixed_tp8/decode")


def test_tp4_chat_shard_sampled():
    sc = S.ALL["decode_chat_tp4"]()
    log(f"case: decode_chat_tp4 seed={sc.seed} Hq={sc.hq} Hkv={sc.hkv}")
    run = ScenarioRun(sc)
    inp, _, od = run_phase(run, 0)
    lens = np.array([l for _, l in inp.dec_meta])
    check_decode(run, inp, od, sample=sorted({int(lens.argmax()), int(lens.argmin()), 9, 200}),
                 what="decode_chat_tp4")


def test_tp4_branching_shard_two_phases():
    sc = S.ALL["branching_tp4"]()
    log(f"case: branching_tp4 seed={sc.seed} Hq={sc.hq} Hkv={sc.hkv}")
    run = ScenarioRun(sc)
    inp, oe, _ = run_phase(run, 0)
    check_extend(run, inp, oe, sample=[0, 63], rows_per_req=16, what="branching_tp4/extend")
    run.finish(0, inp)
    inp2, _, od = run_phase(run, 1)
    check_decode(run, inp2, od, sample=[0, 33, 63], what="branching_tp4/decode")
