"""Seeded input generators (CPU only): definitions, determinism, recipe shapes."""
import numpy as np
import pytest

from workload import contentgen as cg
from workload import scenarios as S


def test_splitmix64_reference_outputs():
    # SplitMix64 seeded with 0 (state += GAMMA, then mix): first outputs as
    # published with the generator's reference code.
    got = [int(cg.splitmix64_nth(0, n)) for n in (1, 2, 3)]
    assert got == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_bf16_round_to_nearest_even():
    f = np.array([1.0, 1.00390625, 1.01171875, 1.0 + 2.0**-8 + 2.0**-20, -2.5, 0.0,
                  -1.00390625], dtype=np.float32)
    assert cg.f32_to_bf16_bits_rne(f).tolist() == [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC020, 0x0000, 0xBF80]


def test_c_and_numpy_generators_agree_bit_for_bit():
    if cg._lib() is None:
        pytest.skip("libcontentgen.so not built")
    rng = np.random.default_rng(0)
    toks = rng.integers(0, S.VOCAB, size=3000).astype(np.int32)
    h = cg.prefix_hashes(toks, 5)
    assert np.array_equal(h, cg.prefix_hashes_np(toks, 5))
    for stream in (cg.STREAM_K, cg.STREAM_V, cg.STREAM_Q):
        assert np.array_equal(cg.values_bf16_bits(h[:200], stream, 512),
                              cg.values_bf16_bits_np(h[:200], stream, 512))
    assert np.array_equal(cg.run_tokens(77, 999, S.VOCAB), cg.run_tokens_np(77, 999, S.VOCAB))


def test_values_are_unit_normal_like_and_exact_bf16():
    h = cg.prefix_hashes(np.arange(4000, dtype=np.int32), 3)
    v = cg.values(h, cg.STREAM_K, 2, 128)
    assert abs(v.mean()) < 0.01 and abs(v.std() - 1.0) < 0.01
    assert np.abs(v).max() <= 6.0
    bits = v.view(np.uint32)
    assert np.all(bits & 0xFFFF == 0)  # representable in bf16


def test_prefix_hash_depends_on_whole_prefix():
    a = np.array([5, 6, 7, 8], dtype=np.int32)
    b = np.array([9, 6, 7, 8], dtype=np.int32)
    ha, hb = cg.prefix_hashes(a, 1), cg.prefix_hashes(b, 1)
    assert not np.any(ha == hb)
    assert np.array_equal(cg.prefix_hashes(a[:2], 1), ha[:2])
    batch = cg.prefix_hashes_batch([a, b, a[:3]], 1)
    assert np.array_equal(batch[0], ha) and np.array_equal(batch[1], hb) and np.array_equal(batch[2], ha[:3])


def test_recipes_are_deterministic():
    for name in ("decode_tiny", "decode_chat", "mixed_small"):
        a, b = S.ALL[name](), S.ALL[name]()
        for pa, pb in zip(a.phases, b.phases):
            for ra, rb in zip(pa.decode + pa.extend, pb.decode + pb.extend):
                assert np.array_equal(ra.tokens, rb.tokens)
        assert np.array_equal(a.free_order(), b.free_order())


def test_recipe_shapes():
    c1 = S.cfg1_decode_tiny()
    assert (c1.hq, c1.hkv, c1.d, c1.pool_slots) == (8, 8, 64, 1024)
    assert all(144 <= r.seq_len <= 192 for r in c1.phases[0].decode)
    c2 = S.cfg2_extend_fewshot()
    assert [(r.prefix_len, r.extend_len) for r in c2.phases[0].extend] == [(2048, 128)] * 64
    c3 = S.cfg3_decode_chat()
    assert len(c3.phases[0].decode) == 256 and all(512 <= r.seq_len <= 4096 for r in c3.phases[0].decode)
    c4 = S.cfg4_branching()
    assert [r.prefix_len for r in c4.phases[0].extend] == [8704] * 64
    assert [r.seq_len for r in c4.phases[1].decode] == [8769] * 64
    for e, d in zip(c4.phases[0].extend, c4.phases[1].decode):
        assert np.array_equal(d.tokens[:8768], e.tokens)


@pytest.mark.slow
def test_mixed_fits_pool():
    sc = S.cfg5_mixed()
    ph = sc.phases[0]
    assert len(ph.extend) == 32 and len(ph.decode) == 512
    assert all(1024 <= r.prefix_len <= 8192 and 256 <= r.extend_len <= 2048 for r in ph.extend)
    assert all(1024 <= r.seq_len <= 16384 for r in ph.decode)
    assert S.unique_context_tokens(sc) <= 0.9 * sc.pool_slots


def test_jump_forward_and_shard_recipes():
    jf = S.jump_forward()
    ph = jf.phases[0]
    assert len(ph.extend) == 256 and (jf.hq, jf.hkv, jf.d) == (32, 8, 128)
    assert all(1024 <= r.prefix_len <= 8192 and 2 <= r.extend_len <= 32 for r in ph.extend)
    assert all(len(r.tokens) == r.prefix_len + r.extend_len for r in ph.extend)
    assert S.unique_context_tokens(jf) <= 0.9 * jf.pool_slots
    # a head shard keeps every request and token of its base workload
    for shard, base, heads in (("decode_chat_tp4", S.cfg3_decode_chat, (8, 2)),
                               ("branching_tp4", S.cfg4_branching, (8, 2))):
        a, b = S.ALL[shard](), base()
        assert (a.hq, a.hkv) == heads and a.seed == b.seed and a.pool_slots == b.pool_slots
        for pa_, pb_ in zip(a.phases, b.phases):
            for ra, rb in zip(pa_.decode + pa_.extend, pb_.decode + pb_.extend):
                assert np.array_equal(ra.tokens, rb.tokens)


def test_bench_work_accounting_and_bound():
    """bench.py's algorithmic work: flops over unmasked pairs, per-request
    and distinct-row bytes, and the roofline bound picked from intensity."""
    import importlib.util
    import os
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(root, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    argv, sys.argv = sys.argv, ["bench"]
    try:
        spec.loader.exec_module(bench)
    finally:
        sys.argv = argv

    class Inp:
        pass

    sc = S.cfg2_extend_fewshot()
    inp = Inp()
    inp.ext_meta = [(r.tokens, r.prefix_len, r.extend_len, 0) for r in sc.phases[0].extend]
    inp.dec_meta, inp.n_dec = [], 0
    w = bench.algorithmic_work(sc, inp)
    # 64 requests x 32 heads x 4 D flops per unmasked (query, key) pair
    assert w["pairs"] == 64 * (128 * 2048 + 128 * 129 // 2)
    assert w["ext_flops"] == 4.0 * 128 * 32 * w["pairs"]
    # distinct rows: the shared 2048-token prefix once, each request's 128 new tokens
    row = 2 * 32 * 128 * 2
    assert w["ext_unique_bytes"] == (2048 + 64 * 128) * row + 64 * 128 * 2 * 32 * 128 * 2
    ridge = bench.BF16_PEAK_TFLOPS * 1e12 / (bench.HBM_PEAK_GBS * 1e9)
    assert w["ext_flops"] / w["ext_unique_bytes"] > ridge      # few-shot extend: MFMA-bound
    jf = S.jump_forward(n_req=16)
    inp2 = Inp()
    inp2.ext_meta = [(r.tokens, r.prefix_len, r.extend_len, 0) for r in jf.phases[0].extend]
    inp2.dec_meta, inp2.n_dec = [], 0
    w2 = bench.algorithmic_work(jf, inp2)
    assert w2["ext_flops"] / w2["ext_unique_bytes"] < ridge    # short extends: HBM-bound
