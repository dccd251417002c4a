"""MFMA wait states of the extend kernel, checked on its gfx950 assembly.

The extend kernel issues its MFMAs from inline assembly, for which the
compiler inserts no wait states; a missing one gives wrong values only now
and then.  These CPU tests compile extend.hip with the library's own flags to
assembly and run tests/mfma_hazards.py over every instantiated kernel, and
check the checker itself on small hand-written sequences.
"""
from __future__ import annotations

import importlib.util
import os
import shutil
import subprocess

import pytest

from tests import mfma_hazards as H

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _build_lib():
    path = os.path.join(ROOT, "paper_2312_07104_amd", "build_lib.py")
    spec = importlib.util.spec_from_file_location("_radixattn_build_lib_hz", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _asm(tmp_path, src_name: str) -> str:
    bl = _build_lib()
    if not os.path.exists(bl.HIPCC) and not shutil.which(bl.HIPCC):
        pytest.skip("hipcc not available")
    src = os.path.join(bl.CSRC, src_name)
    out = tmp_path / (src_name + ".s")
    cmd = [bl.HIPCC, *bl.COMMON, *bl.HIP_ONLY, *bl.EXTRA.get(src_name, []), "--cuda-device-only", "-S", src,
           "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return out.read_text()


def test_extend_kernels_keep_mfma_wait_states(tmp_path):
    ks = {n: b for n, b in H.kernels(_asm(tmp_path, "extend.hip")).items() if "extend_kernel" in n}
    assert len(ks) == 4, sorted(ks)  # <D, waves, tile> for D in {64, 128}, two shapes each
    found = {}
    for name, body in ks.items():
        ins = H.parse(body)
        assert sum(i.mfma for i in ins) > 0
        hz = H.check(ins)
        if hz:
            found[name] = hz[:5]
    assert not found, found


def _seq(*lines):
    return H.check(H.parse(list(lines)))


def test_checker_flags_mfma_result_read_too_early():
    mfma = "v_mfma_f32_16x16x32_bf16 v[10:13], v[2:5], a[0:3], v[10:13]"
    assert _seq(mfma, "v_max_f32_e32 v1, v10, v11", "s_endpgm")
    assert _seq(mfma, "s_nop 5", "v_max_f32_e32 v1, v12, v11", "s_endpgm")
    assert not _seq(mfma, "s_nop 7", "s_nop 2", "v_max_f32_e32 v1, v10, v11", "s_endpgm")
    # unrelated registers are fine
    assert not _seq(mfma, "v_max_f32_e32 v1, v20, v21", "s_endpgm")
    # accumulation chain into the same range is forwarded, a partial overlap is not
    assert not _seq(mfma, "v_mfma_f32_16x16x32_bf16 v[10:13], v[6:9], a[4:7], v[10:13]", "s_endpgm")
    assert _seq(mfma, "v_mfma_f32_16x16x32_bf16 v[20:23], v[10:13], a[4:7], v[20:23]", "s_endpgm")


def test_checker_uses_the_longer_waits_of_32x32_mfmas():
    mfma = "v_mfma_f32_32x32x16_bf16 v[10:25], v[2:5], a[0:3], v[10:25]"
    # 11 wait states cover a 16x16x32 MFMA but not a 32x32x16 one
    assert _seq(mfma, "s_nop 7", "s_nop 2", "v_max_f32_e32 v1, v20, v11", "s_endpgm")
    assert not _seq(mfma, "s_nop 7", "s_nop 3", "v_max_f32_e32 v1, v20, v11", "s_endpgm")
    assert _seq(mfma, "s_nop 7", "s_nop 2", "v_mfma_f32_32x32x16_bf16 v[30:45], v[10:13], a[0:3], 0", "s_endpgm")
    # the C-operand read lasts longer too
    war = "v_mfma_f32_32x32x16_bf16 v[30:45], v[2:5], a[0:3], v[10:25]"
    assert _seq(war, "s_nop 7", "v_mov_b32_e32 v12, 0", "s_endpgm")
    assert not _seq(war, "s_nop 7", "s_nop 2", "v_mov_b32_e32 v12, 0", "s_endpgm")


def test_checker_reads_past_early_exits():
    # a kernel body does not end at its first s_endpgm
    text = "\n".join([
        "\t.type\tk,@function", "k:", "\ts_cbranch_scc1 .LBB0_2", "\ts_endpgm", ".LBB0_2:",
        "\tv_mfma_f32_32x32x16_bf16 v[10:25], v[2:5], a[0:3], v[10:25]", "\tv_max_f32_e32 v1, v10, v11",
        "\ts_endpgm", ".Lfunc_end0:"])
    body = H.kernels(text)["k"]
    assert H.check(H.parse(body))


def test_checker_flags_valu_write_then_mfma_read():
    assert _seq("v_mov_b32_e32 v3, 0", "v_mfma_f32_16x16x32_bf16 v[10:13], v[2:5], a[0:3], 0", "s_endpgm")
    assert _seq("v_accvgpr_write_b32 a2, v7", "v_mfma_f32_16x16x32_bf16 v[10:13], v[2:5], a[0:3], 0", "s_endpgm")
    assert not _seq("v_mov_b32_e32 v3, 0", "s_nop 1", "v_mfma_f32_16x16x32_bf16 v[10:13], v[2:5], a[0:3], 0",
                    "s_endpgm")


def test_checker_flags_accumulator_input_overwritten():
    mfma = "v_mfma_f32_16x16x32_bf16 v[10:13], v[2:5], a[0:3], v[6:9]"
    assert _seq(mfma, "ds_read_b128 v[6:9], v1 offset:16", "s_endpgm")
    assert not _seq(mfma, "s_nop 6", "ds_read_b128 v[6:9], v1 offset:16", "s_endpgm")


def test_checker_follows_loop_back_edges():
    # the read at the loop head comes right after the MFMA at the loop end
    body = [".LBB0_1:", "v_max_f32_e32 v1, v10, v11", "s_nop 3",
            "v_mfma_f32_16x16x32_bf16 v[10:13], v[2:5], a[0:3], v[10:13]", "s_cbranch_scc1 .LBB0_1", "s_nop 7",
            "s_nop 7", "s_endpgm"]
    hz = H.check(H.parse(body))
    assert any("v_max_f32" in h for h in hz)
