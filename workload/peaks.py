"""Measured machine peaks for the roofline report (HIP kernels in csrc/peaks.hip).

* ``hbm_read_gbs``: a streaming read of a 4 GiB buffer (16-byte loads).
* ``gather256_gbs``: 16M random 256-byte head rows of an 8 GiB pool of
  2 KiB slots (8 heads x 128 x bf16), the access pattern of decode over a
  pool of one-token pages.
* ``gather_kv_gbs``: the same rows read as the decode kernels read them:
  K and V rows of one head from two 8 GiB pools in 32-row tiles, 64 bytes of
  16 rows per wave instruction, two tiles in flight, one wave per SIMD
  (8M random rows).
* ``mfma16_bf16_tflops`` / ``mfma32_bf16_tflops``: loops of 16x16x32 and
  32x32x16 bf16 MFMAs, eight independent chains per wave, one wave per SIMD;
  with the cycles per instruction and the shader clock each wave measured.

Each figure is the median of several launches timed with HIP events on the
stream the kernels run on.  No attention is computed here.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpeaks.so")


def _lib():
    if not os.path.exists(_PATH):
        raise ImportError(f"{_PATH} is missing; run __graft_entry__.build()")
    lib = ctypes.CDLL(_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    lib.pk_read.argtypes = [vp, i64, vp, i32, vp]
    lib.pk_gather.argtypes = [vp, vp, i64, i32, i32, vp, i32, vp]
    lib.pk_gather_kv.argtypes = [vp, vp, vp, i32, i32, vp, i32, vp]
    lib.pk_mfma.argtypes = [i32, i32, vp, vp, i32, vp]
    for f in (lib.pk_read, lib.pk_gather, lib.pk_gather_kv, lib.pk_mfma):
        f.restype = ctypes.c_int
    return lib


def _timed(launch, reps: int) -> float:
    """Median milliseconds of `launch()` over reps launches (after two warm-ups)."""
    import torch

    s = torch.cuda.current_stream()
    for _ in range(2):
        launch(s)
    ts = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        launch(s)
        b.record(s)
        b.synchronize()
        ts.append(a.elapsed_time(b))
    return float(np.median(ts))


def measure(reps: int = 7, read_gib: int = 4, pool_gib: int = 8, gather_rows: int = 1 << 24,
            mfma_iters: int = 20000) -> dict:
    import torch

    lib = _lib()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    dev = "cuda"

    def chk(rc):
        if rc != 0:
            raise RuntimeError("peak microbenchmark launch failed")

    out = {}
    blocks = cus * 8
    sink = torch.empty(blocks * 256, dtype=torch.int32, device=dev)
    nbytes = read_gib << 30
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device=dev)
    ms = _timed(lambda s: chk(lib.pk_read(buf.data_ptr(), nbytes, sink.data_ptr(), blocks, s.cuda_stream)), reps)
    out["hbm_read_gbs"] = nbytes / (ms * 1e-3) / 1e9
    del buf

    slot_bytes, heads = 2048, 8
    n_slots = (pool_gib << 30) // slot_bytes
    pool = torch.ones((pool_gib << 30) // 4, dtype=torch.int32, device=dev)
    slots = torch.from_numpy(np.random.default_rng(0).integers(0, n_slots, gather_rows, dtype=np.int32)).to(dev)
    ms = _timed(lambda s: chk(lib.pk_gather(pool.data_ptr(), slots.data_ptr(), gather_rows, heads, slot_bytes,
                                            sink.data_ptr(), blocks, s.cuda_stream)), reps)
    out["gather256_gbs"] = gather_rows * 256 / (ms * 1e-3) / 1e9
    del pool, slots

    # decode tile pattern: one 256-thread work-group per CU, 64 tiles of 32 rows per wave
    kv_blocks, kv_tiles = cus, 64
    kv_rows = kv_blocks * 4 * kv_tiles * 32
    kpool = torch.ones((pool_gib << 30) // 4, dtype=torch.int32, device=dev)
    vpool = torch.ones((pool_gib << 30) // 4, dtype=torch.int32, device=dev)
    slots = torch.from_numpy(np.random.default_rng(1).integers(0, n_slots, kv_rows, dtype=np.int32)).to(dev)
    ms = _timed(lambda s: chk(lib.pk_gather_kv(kpool.data_ptr(), vpool.data_ptr(), slots.data_ptr(), kv_tiles,
                                               slot_bytes, sink.data_ptr(), kv_blocks, s.cuda_stream)), reps)
    out["gather_kv_gbs"] = kv_rows * 512 / (ms * 1e-3) / 1e9
    del kpool, vpool, slots

    mblocks = cus  # one 256-thread work-group per CU: one wave per SIMD
    fsink = torch.empty(mblocks * 256, dtype=torch.float32, device=dev)
    clocks = torch.zeros((mblocks * 4, 2), dtype=torch.int64, device=dev)
    for shape, flops in ((16, 16 * 16 * 32 * 2), (32, 32 * 32 * 16 * 2)):
        ms = _timed(lambda s: chk(lib.pk_mfma(shape, mfma_iters, fsink.data_ptr(), clocks.data_ptr(), mblocks,
                                              s.cuda_stream)), reps)
        total = mblocks * 4 * mfma_iters * 8 * flops
        out[f"mfma{shape}_bf16_tflops"] = total / (ms * 1e-3) / 1e12
        c = clocks.cpu().numpy().astype(np.float64)
        out[f"mfma{shape}_cycles_per_instr"] = float(np.median(c[:, 0]) / (8 * mfma_iters))
        out[f"mfma{shape}_shader_ghz"] = float(np.median(c[:, 0] / (c[:, 1] / 100e6)) / 1e9)
    torch.cuda.synchronize()
    return out
