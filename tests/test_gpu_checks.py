"""Device-side batch validation (ra_check_batch, ra_set_debug_checks).

Planted faults in copies of a valid batch's device arrays (slots outside the
pool, table rows outside the table, lengths past their bounds) are reported
with the request, the field and the position; with the debug switch on the
attention calls refuse such a batch before launching anything (their outputs
stay untouched) and run a valid one unchanged.  Nothing here launches an
attention kernel on a bad batch.
"""
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU-only container
    pytest.skip("no GPU", allow_module_level=True)

import paper_2312_07104_amd as pa  # noqa: E402
from tests.harness import ScenarioRun, log, make_scenario  # noqa: E402


@pytest.fixture(scope="module")
def batch():
    sc = make_scenario("checks", 16, 4, 128, 8192, extend=[(300, 40), (0, 17), (700, 5)], decode=[500, 1, 1200],
                       seed=61)
    run = ScenarioRun(sc)
    inp = run.prepare(0)
    run.store(inp)
    torch.cuda.synchronize()
    return run, inp


def _ext(run, inp, table=None, rpi=None, prefix=None, elen=None, start=None, max_e=None):
    pa.ra_check_batch(inp.table if table is None else table, inp.rpi[: inp.n_ext] if rpi is None else rpi,
                      run.sc.pool_slots, inp.prefix_lens if prefix is None else prefix,
                      inp.extend_lens if elen is None else elen, inp.extend_start if start is None else start,
                      inp.total_ext, inp.max_extend_len if max_e is None else max_e)


def _dec(run, inp, table=None, rpi=None, lens=None):
    pa.ra_check_batch(inp.table if table is None else table, inp.rpi[inp.n_ext:] if rpi is None else rpi,
                      run.sc.pool_slots, seq_lens=inp.seq_lens if lens is None else lens,
                      max_seq_len=inp.max_seq_len)


def test_valid_batch_passes(batch):
    run, inp = batch
    log("case: checks on a valid batch")
    _ext(run, inp)
    _dec(run, inp)


@pytest.mark.parametrize("what", ["slot_high", "slot_negative", "decode_slot", "row", "seq_len", "seq_len_zero",
                                  "extend_len", "extend_start", "prefix_len"])
def test_planted_fault_is_reported(batch, what):
    run, inp = batch
    log(f"case: planted fault {what}")
    rpi_e, rpi_d = inp.rpi[: inp.n_ext], inp.rpi[inp.n_ext:]
    t = inp.table.clone()
    if what == "slot_high":
        t[rpi_e[2], 123] = run.sc.pool_slots + 5
        with pytest.raises(pa.RadixAttnError, match="request 2: slot outside .* at position 123"):
            _ext(run, inp, table=t)
    elif what == "slot_negative":
        t[rpi_e[0], 299] = -1
        with pytest.raises(pa.RadixAttnError, match="request 0: slot outside .* at position 299"):
            _ext(run, inp, table=t)
    elif what == "decode_slot":
        t[rpi_d[2], 1199] = run.sc.pool_slots  # the query's own slot
        t[rpi_d[2], 999] = run.sc.pool_slots + 1
        with pytest.raises(pa.RadixAttnError, match="request 2: slot outside .* at position 999"):
            _dec(run, inp, table=t)
        # a bad entry past the request's context is never read: not a fault
        t2 = inp.table.clone()
        t2[rpi_d[1], 5] = -7
        _dec(run, inp, table=t2)
    elif what == "row":
        r = rpi_d.clone()
        r[1] = inp.table.shape[0]
        with pytest.raises(pa.RadixAttnError, match="request 1: req_pool_idx"):
            _dec(run, inp, rpi=r)
    elif what in ("seq_len", "seq_len_zero"):
        lens = inp.seq_lens.clone()
        lens[0] = inp.max_seq_len + 1 if what == "seq_len" else 0
        with pytest.raises(pa.RadixAttnError, match="request 0: seq_lens"):
            _dec(run, inp, lens=lens)
    elif what == "extend_len":
        with pytest.raises(pa.RadixAttnError, match="request 0: extend_lens"):
            _ext(run, inp, max_e=inp.max_extend_len - 1)
    elif what == "extend_start":
        s = inp.extend_start.clone()
        s[2] = inp.total_ext - 1
        with pytest.raises(pa.RadixAttnError, match="request 2: extend_start"):
            _ext(run, inp, start=s)
    elif what == "prefix_len":
        p = inp.prefix_lens.clone()
        p[1] = inp.table.shape[1] + 1
        with pytest.raises(pa.RadixAttnError, match="request 1: prefix_lens"):
            _ext(run, inp, prefix=p)


def test_debug_switch_guards_attention_calls(batch):
    run, inp = batch
    log("case: debug switch")
    rpi_d = inp.rpi[inp.n_ext:]
    ref_e = run.extend(inp)
    ref_d = run.decode(inp)
    torch.cuda.synchronize()
    bad = inp.table.clone()
    bad[rpi_d[0], 17] = run.sc.pool_slots + 3
    pa.ra_set_debug_checks(True)
    try:
        out_d = torch.full_like(inp.q_dec, 5.0)
        with pytest.raises(pa.RadixAttnError, match="request 0: slot outside"):
            pa.ra_decode_attention(inp.q_dec, run.k_pool, run.v_pool, bad, rpi_d, inp.seq_lens, inp.max_seq_len,
                                   run.sc.scale, out=out_d)
        with pytest.raises(pa.RadixAttnError, match="request 0: slot outside"):
            pa.ra_decode_attention_noalloc(inp.q_dec, run.k_pool, run.v_pool, bad, rpi_d, inp.seq_lens,
                                           inp.max_seq_len, run.sc.scale, out_d)
        out_e = torch.full_like(inp.q_ext, 5.0)
        with pytest.raises(pa.RadixAttnError, match="request 0: slot outside"):
            pa.ra_mixed_attention(inp.q_ext, inp.k_new[: inp.total_ext], inp.v_new[: inp.total_ext],
                                  inp.rpi[: inp.n_ext], inp.prefix_lens, inp.extend_lens, inp.extend_start,
                                  inp.max_extend_len, inp.q_dec, rpi_d, inp.seq_lens, inp.max_seq_len, run.k_pool,
                                  run.v_pool, bad, run.sc.scale, out_ext=out_e, out_dec=out_d)
        torch.cuda.synchronize()
        assert bool((out_d == 5.0).all()) and bool((out_e == 5.0).all())
        # a valid batch runs as without the switch
        me, md = run.mixed(inp)
        torch.cuda.synchronize()
        assert torch.equal(me, ref_e) and torch.equal(md, ref_d)
    finally:
        pa.ra_set_debug_checks(False)
