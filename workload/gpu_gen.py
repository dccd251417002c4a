"""GPU fill of content-addressed values (the HIP twin of contentgen.values).

Writes bf16 rows straight into device tensors so multi-gigabyte KV pools can
be filled without host staging.  Input generation only.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libworkgen.so")
_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_PATH):
            raise ImportError(f"{_PATH} is missing; run __graft_entry__.build()")
        _LIB = ctypes.CDLL(_PATH)
        _LIB.wg_values.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                   ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
        _LIB.wg_values.restype = ctypes.c_int
    return _LIB


def fill(out, hashes: np.ndarray, stream: int, rows: np.ndarray | None = None, scale_pow2: int = 0,
         chunk: int = 1 << 18) -> None:
    """out[rows[p]] (or out[p]) = values(hashes[p]); out is a bf16 CUDA tensor
    whose trailing dimensions hold one position's elements."""
    import torch

    n_elem = int(np.prod(out.shape[1:]))
    h_all = np.ascontiguousarray(hashes, dtype=np.uint64)
    r_all = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    if r_all is not None and r_all.size and (r_all.min() < 0 or r_all.max() >= out.shape[0]):
        raise IndexError("fill rows outside the output tensor")
    if r_all is None and h_all.shape[0] > out.shape[0]:
        raise IndexError("more positions than output rows")
    s = torch.cuda.current_stream().cuda_stream
    for a in range(0, h_all.shape[0], chunk):
        h = torch.from_numpy(h_all[a : a + chunk].view(np.int64)).to(out.device)
        if r_all is None:
            r = None
            base = out[a:]
        else:
            r = torch.from_numpy(r_all[a : a + chunk]).to(out.device)
            base = out
        rc = lib().wg_values(ctypes.c_void_p(h.data_ptr()), None if r is None else ctypes.c_void_p(r.data_ptr()),
                             h.shape[0], stream, n_elem, scale_pow2, ctypes.c_void_p(base.data_ptr()),
                             ctypes.c_void_p(s))
        if rc != 0:
            raise RuntimeError("wg_values launch failed")
        torch.cuda.current_stream().synchronize()  # keep h / r alive until the kernel is done
