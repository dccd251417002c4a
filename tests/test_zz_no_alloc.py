"""The allocation-free decode entry point against the workspace one.

Two calls in a row through ra_decode_attention_noalloc (the second with a
smaller batch, so it runs over what the first left in the shared scratch)
must equal ra_decode_attention with a caller workspace bit for bit (same
kernels, same chunking) and match the oracle; torch's allocator must see no
allocation during the calls; a batch whose split partials exceed the scratch
is rejected before anything is launched.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only container
    pytest.skip("no GPU", allow_module_level=True)

import paper_2312_07104_amd as pa  # noqa: E402
from oracle import attention as oa  # noqa: E402
from tests.harness import ScenarioRun, assert_close, log, make_scenario  # noqa: E402


def _batch(seed, lens, hq=32, hkv=8):
    sc = make_scenario(f"noalloc{seed}", hq, hkv, 128, sum(lens) + 256, decode=lens, seed=seed)
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    torch.cuda.synchronize()
    return run, inp


def _allocs():
    return torch.cuda.memory_stats().get("allocation.all.allocated", 0)


def test_noalloc_decode_matches_workspace_entry_point():
    rng = np.random.default_rng(3)
    big = [int(x) for x in rng.integers(1, 6000, 48)] + [6000, 4096, 1]
    small = [int(x) for x in rng.integers(1, 1500, 9)] + [2047]
    cases = [_batch(201, big), _batch(202, small)]
    outs = []
    for run, inp in cases:
        out = torch.full_like(inp.q_dec, 3.0)
        outs.append(out)
    for (run, inp), out in zip(cases, outs):
        need = pa.ra_decode_workspace_bytes(inp.n_dec, run.sc.hq, run.sc.hkv, run.sc.d, inp.max_seq_len)
        log(f"case: noalloc decode batch={inp.n_dec} max_len={inp.max_seq_len} scratch={need}")
        assert 0 < need <= pa.ra_decode_noalloc_max_scratch_bytes()
        n0 = _allocs()
        pa.ra_decode_attention_noalloc(inp.q_dec, run.k_pool, run.v_pool, inp.table, inp.rpi, inp.seq_lens,
                                       inp.max_seq_len, run.sc.scale, out)
        assert _allocs() == n0
    torch.cuda.synchronize()
    for (run, inp), out in zip(cases, outs):
        ref = run.decode(inp)  # the workspace entry point
        torch.cuda.synchronize()
        assert torch.equal(out, ref)
        got = out.float().cpu().numpy()
        sc = run.sc
        for i in range(0, inp.n_dec, 7):
            toks, L = inp.dec_meta[i]
            assert_close(got[i], oa.decode_reference(toks, L, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale),
                         f"noalloc decode req {i} L={L}")


def test_noalloc_decode_rejects_oversized_batch():
    b, hq, hkv, d, max_len, splits = 64, 64, 8, 128, 16384, 512
    need = pa.ra_decode_workspace_bytes(b, hq, hkv, d, max_len, splits)
    log(f"case: noalloc oversized scratch={need}")
    assert need > pa.ra_decode_noalloc_max_scratch_bytes()
    q = torch.zeros((b, hq, d), dtype=torch.bfloat16, device="cuda")
    pool = torch.zeros((64, hkv, d), dtype=torch.bfloat16, device="cuda")
    table = torch.zeros((b, max_len), dtype=torch.int32, device="cuda")
    rpi = torch.arange(b, dtype=torch.int32, device="cuda")
    lens = torch.full((b,), max_len, dtype=torch.int32, device="cuda")
    out = torch.full_like(q, 7.0)
    with pytest.raises(pa.RadixAttnError, match="scratch"):
        pa.ra_decode_attention_noalloc(q, pool, pool, table, rpi, lens, max_len, 0.088, out, num_splits=splits)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
