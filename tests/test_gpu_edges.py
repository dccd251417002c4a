"""GPU edge cases: degenerate lengths, ragged tiles, chunk boundaries, needles,
sharpened scores, slot-permutation invariance, reuse versus recomputation."""
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
from tests.harness import ScenarioRun, assert_close, log  # noqa: E402
from tests.harness import make_scenario as _scenario  # noqa: E402
from workload import gpu_gen  # noqa: E402


def _bf(t):
    return t.float().cpu().numpy()


def _run(sc, num_splits=0):
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    oe = run.extend(inp)
    od = run.decode(inp, num_splits=num_splits)
    torch.cuda.synchronize()
    return run, inp, oe, od


def _check_all(run, inp, oe, od, what):
    sc = run.sc
    if oe is not None:
        got = _bf(oe)
        for toks, p, e, start in inp.ext_meta:
            if e == 0:
                continue
            ref = oa.extend_reference(toks, p, e, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale, sc.q_scale_pow2)
            assert_close(got[start:start + e], ref, f"{what} extend P={p} E={e}")
    if od is not None:
        got = _bf(od)
        for i, (toks, l) in enumerate(inp.dec_meta):
            ref = oa.decode_reference(toks, l, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale, sc.q_scale_pow2)
            assert_close(got[i], ref, f"{what} decode L={l}")


@pytest.mark.parametrize("hq,hkv,d", [(8, 8, 64), (32, 8, 128), (16, 1, 128), (6, 2, 64)])
def test_single_key_returns_v_exactly(hq, hkv, d):
    log(f"case: single key hq={hq} hkv={hkv} d={d}")
    ext = [(0, 1)] if (hq // hkv) in (1, 2, 4, 8, 16) else []
    sc = _scenario("single", hq, hkv, d, 64, extend=ext, decode=[1, 1])
    run, inp, oe, od = _run(sc)
    v = run.v_pool.float().cpu().numpy()
    for i, (toks, l) in enumerate(inp.dec_meta):
        slot = inp.plan.rows[inp.n_ext + i][0]
        for h in range(hq):
            assert np.array_equal(_bf(od)[i, h], v[slot, h // (hq // hkv)])
    if oe is not None:
        slot = inp.plan.rows[0][0]
        for h in range(hq):
            assert np.array_equal(_bf(oe)[0, h], v[slot, h // (hq // hkv)])


@pytest.mark.parametrize("hq,hkv,d", [(8, 8, 64), (32, 8, 128), (64, 8, 128), (16, 1, 64), (32, 2, 128)])
def test_ragged_extend_tiles(hq, hkv, d):
    log(f"case: ragged extend hq={hq} hkv={hkv} d={d}")
    ext = [(0, 1), (5, 130), (64, 63), (63, 65), (0, 200), (130, 7), (1, 0), (257, 129)]
    sc = _scenario("ragged", hq, hkv, d, 4096, extend=ext, seed=hq + d)
    run, inp, oe, od = _run(sc)
    _check_all(run, inp, oe, od, "ragged")


@pytest.mark.parametrize("hq,hkv,d", [(8, 8, 64), (8, 8, 128), (16, 4, 128), (32, 8, 64)])
def test_extend_kernels_agree_with_oracle(hq, hkv, d):
    """The same batch through the 128-row kernel (query rows per kv head below
    256) and through the 256-row kernel (forced by an inflated, still valid,
    upper bound on the extend length, large enough that the 256-row launch
    has at least one work-group per CU; the extra work-groups have no rows
    and end at once): both match the oracle."""
    log(f"case: both extend kernels hq={hq} hkv={hkv} d={d}")
    grp = hq // hkv
    e_max = max(1, 255 // grp)  # largest extend that stays on the 128-row kernel
    ext = [(0, e_max), (70, max(1, e_max // 3)), (129, 1), (300, max(1, e_max - 5)), (64, 64 // grp or 1)]
    sc = _scenario("two-kernels", hq, hkv, d, 4096, extend=ext, seed=31 + hq + d)
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    assert inp.max_extend_len * grp < 256
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    tpb = 256 // grp  # new tokens per 256-row work-group
    wide = max(inp.max_extend_len, tpb + 1, tpb * -(-cus // (inp.n_ext * hkv)))
    assert inp.n_ext * hkv * -(-wide // tpb) >= cus
    outs = {}
    for name, bound in (("narrow", inp.max_extend_len), ("wide", wide)):
        outs[name] = pa.ra_extend_attention(
            inp.q_ext, inp.k_new[: inp.total_ext], inp.v_new[: inp.total_ext], run.k_pool, run.v_pool, inp.table,
            inp.rpi[: inp.n_ext], inp.prefix_lens, inp.extend_lens, inp.extend_start, bound, sc.scale)
    torch.cuda.synchronize()
    for name, o in outs.items():
        got = _bf(o)
        for toks, p, e, start in inp.ext_meta:
            ref = oa.extend_reference(toks, p, e, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale, sc.q_scale_pow2)
            assert_close(got[start:start + e], ref, f"{name} kernel P={p} E={e}")


@pytest.mark.parametrize("n_req,hq,hkv", [(1016, 8, 2), (1100, 8, 2), (600, 16, 16)])
def test_extend_work_order_batch_sizes(n_req, hq, hkv):
    """Up to 1016 requests the extend kernel starts its work items longest
    first (ranked inside each work-group); above that it keeps the static
    order.  Both sides of the limit, and 16 kv heads (two per XCD), with
    ragged and equal key counts (ties),
    a request with no new tokens, and empty query-tile slots: every output
    row against the oracle."""
    log(f"case: extend work order n_req={n_req}")
    rng = np.random.default_rng(4000 + n_req)
    ext = [(int(rng.integers(0, 48)), int(rng.integers(1, 12))) for _ in range(n_req)]
    ext[3] = ext[5] = (20, 6)  # equal key counts
    ext[7] = (30, 0)           # no new tokens
    ext[9] = (100, 40)         # longest, several query tiles of 128 rows / 4 heads
    pool = sum(p + e for p, e in ext) + 256
    sc = _scenario(f"order{n_req}", hq, hkv, 64, pool, extend=ext, seed=17 + n_req)
    run, inp, oe, od = _run(sc)
    _check_all(run, inp, oe, od, f"order n_req={n_req}")


@pytest.mark.parametrize("n_req", [700, 1600])
def test_decode_large_batches(n_req):
    """Large decode batches over two kv heads: several thousand (split,
    request) items dealt to the XCDs in turn, ragged lengths with exact chunk
    multiples, single tokens and equal lengths: every output against the
    oracle."""
    log(f"case: decode large batch n_req={n_req}")
    rng = np.random.default_rng(5000 + n_req)
    lens = [int(x) for x in rng.integers(1, 700, n_req)]
    lens[1] = lens[2] = 256  # exact chunk multiples, equal lengths
    lens[4] = 1
    lens[6] = 1000
    sc = _scenario(f"dorder{n_req}", 8, 2, 128, sum(lens) + 256, decode=lens, seed=23 + n_req)
    run, inp, oe, od = _run(sc)
    _check_all(run, inp, oe, od, f"decode order n_req={n_req}")


@pytest.mark.parametrize("kind,d", [("ragged", 128), ("full", 128), ("partial", 128), ("ragged", 64)])
def test_decode_longest_first(kind, d):
    """With 2048-token chunks and more items than the chip's wave slots, the
    decode kernel starts the full chunks first and the partial last chunks
    longest first.  Ragged lengths with exact chunk multiples, contexts
    shorter than one chunk and equal lengths; batches of full chunks only
    and of partial chunks only; both partial-pass kernels (D = 128 register
    staging, D = 64 LDS copies): every output against the oracle."""
    log(f"case: decode longest first {kind} d={d}")
    rng = np.random.default_rng(6100)
    if kind == "full":
        lens = [2048 * int(x) for x in rng.integers(1, 3, 128)]
    elif kind == "partial":
        lens = [int(x) for x in rng.integers(1, 2048, 128)]
        lens[0] = 4096  # two full chunks, so num_splits = 2 keeps chunks 2048 long
    else:
        lens = [int(x) for x in rng.integers(1, 4097, 128)]
        lens[0] = lens[1] = 2048
        lens[2] = 4096
        lens[3] = lens[4] = 3000
        lens[5] = 1
    sc = _scenario(f"dlpt_{kind}_{d}", 8, 8, d, sum(lens) + 256, decode=lens, seed=61)
    assert pa.ra_decode_chunk_len(len(lens), 8, max(lens), 2) == 2048
    run, inp, oe, od = _run(sc, num_splits=2)
    _check_all(run, inp, oe, od, "decode longest first")


@pytest.mark.parametrize("num_splits", [0, 1, 3, 16])
def test_decode_boundaries(num_splits):
    lens = [1, 2, 31, 32, 33, 63, 64, 65, 255, 256, 257, 511, 512, 513, 1000, 2049]
    log(f"case: decode boundaries num_splits={num_splits}")
    sc = _scenario("bounds", 32, 8, 128, 16384, decode=lens, seed=5)
    run, inp, oe, od = _run(sc, num_splits=num_splits)
    _check_all(run, inp, oe, od, f"bounds/splits={num_splits}")


@pytest.mark.parametrize("q_pow2", [2, 3])
def test_sharpened_scores(q_pow2):
    """Q ~ N(0, 16 or 64): softmax concentrates on few keys, so any wrong,
    dropped or duplicated key moves the output by O(1)."""
    log(f"case: sharpened q_pow2={q_pow2}")
    sc = _scenario("sharp", 32, 8, 128, 8192, extend=[(300, 77), (0, 129)], decode=[700, 64, 1537], seed=9,
                   q_pow2=q_pow2)
    run, inp, oe, od = _run(sc)
    _check_all(run, inp, oe, od, "sharp")


def test_decode_needles():
    """A key equal to 8x one head's query dominates that head's softmax: the
    output must be that position's V, at tile and chunk boundaries."""
    L = 1100
    sc = _scenario("needle", 16, 4, 128, 4096, decode=[L], seed=21)
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    torch.cuda.synchronize()
    toks, _ = inp.dec_meta[0]
    row = inp.plan.rows[0]
    chunk = pa.ra_decode_chunk_len(1, 4, L, 3)
    k_ref, v_ref, h = oa.request_kv(toks, sc.seed, sc.hkv, sc.d)
    q = cg.values(h[L - 1:L], cg.STREAM_Q, sc.hq, sc.d)[0]
    for j in (0, 31, 32, chunk - 1, chunk, L - 2, L - 1):
        for head in (0, 7, 13):
            log(f"case: needle pos={j} head={head}")
            g = head // 4
            kk = k_ref.copy()
            kk[j, g] = cg.bf16_bits_to_f32(cg.f32_to_bf16_bits_rne(q[head] * 8))
            saved = run.k_pool[row[j], g].clone()
            run.k_pool[row[j], g] = torch.from_numpy(kk[j, g]).to(torch.bfloat16).cuda()
            out = run.decode(inp, num_splits=3)
            torch.cuda.synchronize()
            run.k_pool[row[j], g] = saved
            qq = cg.values(h[L - 1:L], cg.STREAM_Q, sc.hq, sc.d)
            ref = oa.attend(qq, kk, v_ref, np.array([L - 1]), sc.scale)[0]
            got = _bf(out)[0]
            assert_close(got, ref, f"needle {j}/{head}")
            assert np.abs(got[head] - v_ref[j, g]).max() < 0.05


def test_slot_permutation_is_bit_exact():
    sc = S.cfg5_mixed_small()
    log(f"case: slot permutation seed={sc.seed}")
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    oe = run.extend(inp)
    od = run.decode(inp)
    torch.cuda.synchronize()
    perm = torch.from_numpy(np.random.default_rng(3).permutation(sc.pool_slots)).long().cuda()
    k2 = torch.empty_like(run.k_pool)
    v2 = torch.empty_like(run.v_pool)
    k2[perm] = run.k_pool
    v2[perm] = run.v_pool
    t = inp.table.long()
    table2 = torch.where(t >= 0, perm[t.clamp(min=0)], t).int().contiguous()
    run.k_pool, run.v_pool = k2, v2
    inp.table = table2
    oe2 = run.extend(inp)
    od2 = run.decode(inp)
    torch.cuda.synchronize()
    assert torch.equal(oe, oe2) and torch.equal(od, od2)


@pytest.mark.parametrize("hq,hkv,p,e", [(32, 32, 2048, 128), (32, 8, 700, 90), (64, 8, 1500, 600)])
def test_reused_prefix_equals_recompute(hq, hkv, p, e):
    """Extend over a cached prefix read through the table equals extend of the
    whole sequence as new tokens (prefix_len = 0), within tolerance."""
    log(f"case: reuse vs recompute hq={hq} hkv={hkv} P={p} E={e}")
    d, n = 128, p + e
    toks = cg.run_tokens(4242, n, S.VOCAB)
    h = cg.prefix_hashes(toks, 1)
    dev = "cuda"
    q = torch.empty((n, hq, d), dtype=torch.bfloat16, device=dev)
    kn = torch.empty((n, hkv, d), dtype=torch.bfloat16, device=dev)
    vn = torch.empty_like(kn)
    gpu_gen.fill(q, h, cg.STREAM_Q)
    gpu_gen.fill(kn, h, cg.STREAM_K)
    gpu_gen.fill(vn, h, cg.STREAM_V)
    i32 = lambda a: torch.tensor(a, dtype=torch.int32, device=dev)  # noqa: E731
    # recompute: every position is new
    pool = torch.zeros((8, hkv, d), dtype=torch.bfloat16, device=dev)
    full = pa.ra_extend_attention(q, kn, vn, pool, pool, i32([[0]]), i32([0]), i32([0]), i32([n]), i32([0]), n,
                                  1.0 / np.sqrt(d))
    # reuse: the prefix sits in scattered pool slots
    S_ = 4 * n
    slots = np.random.default_rng(0).choice(S_, p, replace=False).astype(np.int32)
    kp = torch.zeros((S_, hkv, d), dtype=torch.bfloat16, device=dev)
    vp = torch.zeros_like(kp)
    pa.ra_store_kv(torch.from_numpy(slots).cuda(), kn[:p].contiguous(), vn[:p].contiguous(), kp, vp)
    part = pa.ra_extend_attention(q[p:].contiguous(), kn[p:].contiguous(), vn[p:].contiguous(), kp, vp,
                                  torch.from_numpy(slots[None]).cuda(), i32([0]), i32([p]), i32([e]), i32([0]), e,
                                  1.0 / np.sqrt(d))
    torch.cuda.synchronize()
    assert_close(_bf(part), _bf(full)[p:].astype(np.float64), "reuse vs recompute")
    ref = oa.attend(cg.values(h[p:], cg.STREAM_Q, hq, d), cg.values(h, cg.STREAM_K, hkv, d),
                    cg.values(h, cg.STREAM_V, hkv, d), np.arange(p, n), 1.0 / np.sqrt(np.float32(d)))
    assert_close(_bf(part), ref, "reuse vs oracle")


def test_empty_and_invalid_arguments():
    log("case: empty batch and argument errors")
    z = torch.zeros((4, 2, 64), dtype=torch.bfloat16, device="cuda")
    t = torch.zeros((1, 4), dtype=torch.int32, device="cuda")
    e = torch.zeros((0,), dtype=torch.int32, device="cuda")
    out = pa.ra_decode_attention(z[:0], z, z, t, e, e, 4, 0.125)
    assert out.shape[0] == 0
    with pytest.raises(pa.RadixAttnError):
        pa.ra_decode_attention(torch.zeros((1, 3, 64), dtype=torch.bfloat16, device="cuda"), z, z, t,
                               torch.zeros(1, dtype=torch.int32, device="cuda"),
                               torch.ones(1, dtype=torch.int32, device="cuda"), 4, 0.125)
    with pytest.raises(pa.RadixAttnError):  # G = 3 not a power of two for extend
        pa.ra_extend_attention(torch.zeros((1, 6, 64), dtype=torch.bfloat16, device="cuda"), z[:1], z[:1], z, z, t,
                               torch.zeros(1, dtype=torch.int32, device="cuda"),
                               torch.zeros(1, dtype=torch.int32, device="cuda"),
                               torch.ones(1, dtype=torch.int32, device="cuda"),
                               torch.zeros(1, dtype=torch.int32, device="cuda"), 1, 0.125)


def test_mixed_call_equals_separate_calls():
    """ra_mixed_attention runs the same kernels on two streams: outputs are
    bit-identical to separate calls, and ordered before later work on the
    caller's stream."""
    sc = S.cfg5_mixed_small()
    log(f"case: mixed call seed={sc.seed}")
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    oe = run.extend(inp)
    od = run.decode(inp)
    torch.cuda.synchronize()
    for rep in range(3):
        me, md = run.mixed(inp)
        s_e, s_d = me.float().sum(), md.float().sum()  # consumers queued on the caller's stream
        torch.cuda.synchronize()
        assert torch.equal(me, oe) and torch.equal(md, od)
        assert torch.isfinite(s_e) and torch.isfinite(s_d)


def test_mixed_call_decode_heavy_equals_separate_calls():
    """One short extend request beside the whole decode batch (the decode
    finishes long after the extend): both outputs equal separate calls bit for
    bit, over repeated calls on one workspace."""
    sc = S.cfg5_mixed_small()
    log(f"case: decode-heavy mixed call seed={sc.seed}")
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    e0 = int(inp.extend_lens[0].item())
    assert e0 > 0
    args_e = (inp.q_ext[:e0], inp.k_new[:e0], inp.v_new[:e0])
    rpi_e, pre_e, len_e = inp.rpi[:1], inp.prefix_lens[:1], inp.extend_lens[:1]
    start_e = torch.zeros(1, dtype=torch.int32, device="cuda")
    oe = pa.ra_extend_attention(*args_e, run.k_pool, run.v_pool, inp.table, rpi_e, pre_e, len_e, start_e, e0,
                                sc.scale)
    od = run.decode(inp)
    torch.cuda.synchronize()
    ws = torch.empty(pa.ra_decode_workspace_bytes(inp.n_dec, sc.hq, sc.hkv, sc.d, inp.max_seq_len),
                     dtype=torch.uint8, device="cuda")
    for rep in range(3):
        me, md = pa.ra_mixed_attention(*args_e, rpi_e, pre_e, len_e, start_e, e0, inp.q_dec, inp.rpi[inp.n_ext:],
                                       inp.seq_lens, inp.max_seq_len, run.k_pool, run.v_pool, inp.table, sc.scale,
                                       workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(me, oe) and torch.equal(md, od), rep


def test_mixed_call_workspace_too_small_is_rejected():
    sc = S.cfg5_mixed_small()
    log("case: mixed call workspace check")
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    torch.cuda.synchronize()
    need = pa.ra_decode_workspace_bytes(inp.n_dec, sc.hq, sc.hkv, sc.d, inp.max_seq_len)
    assert need > 256  # the batch has split contexts
    out_d = torch.full_like(inp.q_dec, 7.0)
    with pytest.raises(pa.RadixAttnError):
        run.mixed(inp, workspace=torch.empty(need - 256, dtype=torch.uint8, device="cuda"), out_dec=out_d)
    torch.cuda.synchronize()
    assert bool((out_d == 7.0).all())


def test_mixed_call_rejects_bad_half_without_side_effects():
    sc = S.cfg5_mixed_small()
    log("case: mixed call argument error")
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    torch.cuda.synchronize()
    out_d = torch.full_like(inp.q_dec, 7.0)
    with pytest.raises(pa.RadixAttnError):
        pa.ra_mixed_attention(inp.q_ext, inp.k_new[: inp.total_ext], inp.v_new[: inp.total_ext],
                              inp.rpi[: inp.n_ext], inp.prefix_lens, inp.extend_lens, inp.extend_start,
                              inp.max_extend_len, inp.q_dec, inp.rpi[inp.n_ext:], inp.seq_lens, inp.max_seq_len,
                              run.k_pool, run.v_pool, inp.table, -1.0, out_dec=out_d)  # negative scale
    torch.cuda.synchronize()
    assert bool((out_d == 7.0).all())


@pytest.mark.parametrize("case", range(24))
def test_random_small_batches(case):
    """Seeded random batches: group sizes, kv-head counts, head sizes, ragged
    prefix / extend / decode lengths and split counts that the fixed cases do
    not list.  Every output against the oracle; where the batch has both
    halves, the mixed call equals the separate calls bit for bit."""
    rng = np.random.default_rng(9000 + case)
    grp = int(rng.choice([1, 2, 4, 8, 16]))
    hkv = int(rng.choice([1, 2, 4, 8]))
    hkv = max(1, min(hkv, 64 // grp))
    hq, d = grp * hkv, int(rng.choice([64, 128]))
    n_ext = int(rng.integers(0, 5))
    n_dec = int(rng.integers(0 if n_ext else 1, 6))
    extend = [(int(rng.integers(0, 700)), int(rng.integers(1, 200))) for _ in range(n_ext)]
    decode = [int(rng.integers(1, 3000)) for _ in range(n_dec)]
    num_splits = int(rng.choice([0, 0, 1, 2, 5, 17]))
    pool = sum(p + e for p, e in extend) + sum(decode) + 256
    log(f"case: random {case} hq={hq} hkv={hkv} d={d} extend={extend} decode={decode} splits={num_splits}")
    sc = _scenario(f"random{case}", hq, hkv, d, pool, extend=extend, decode=decode, seed=300 + case)
    run, inp, oe, od = _run(sc, num_splits=num_splits)
    _check_all(run, inp, oe, od, f"random {case}")
    if n_ext and n_dec:
        me, md = run.mixed(inp, num_splits=num_splits)
        torch.cuda.synchronize()
        assert torch.equal(me, oe) and torch.equal(md, od)
