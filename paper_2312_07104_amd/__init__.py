"""RadixAttention hot path for MI355X (gfx950): Python binding of libradixattn.

Argument marshalling only.  Every step runs in the native library: the host
radix cache in C++, attention and the KV scatter in HIP kernels.  Torch
tensors provide device memory and the current HIP stream.  Importing this
package fails if the native library has not been built (``build_lib.py``).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libradixattn.so")

RA_OK, RA_EINVAL, RA_ENOMEM, RA_EHIP = 0, -1, -2, -3

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python {_HERE}/build_lib.py`")

_lib = ctypes.CDLL(LIB_PATH)

_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int32

_SIGS = {
    "ra_last_error": ([], ctypes.c_char_p),
    "ra_cache_create": ([_i64, _vp, ctypes.POINTER(_vp)], ctypes.c_int),
    "ra_cache_destroy": ([_vp], None),
    "ra_match_prefix": ([_vp, _vp, _i64, _vp, _i64p, _i64p], ctypes.c_int),
    "ra_inc_ref": ([_vp, _i64, _i64p], ctypes.c_int),
    "ra_dec_ref": ([_vp, _i64, _i64p], ctypes.c_int),
    "ra_alloc_slots": ([_vp, _i64, _vp], ctypes.c_int),
    "ra_free_slots": ([_vp, _vp, _i64], ctypes.c_int),
    "ra_insert": ([_vp, _vp, _vp, _i64, _i64p, _i64p], ctypes.c_int),
    "ra_evict": ([_vp, _i64, _i64p], ctypes.c_int),
    "ra_evictable_size": ([_vp], _i64),
    "ra_available_size": ([_vp], _i64),
    "ra_cached_tokens": ([_vp], _i64),
    "ra_num_nodes": ([_vp], _i64),
    "ra_snapshot": ([_vp, _vp, _i64, _i64p], ctypes.c_int),
    "ra_cache_log_evictions": ([_vp, _i32], ctypes.c_int),
    "ra_eviction_log_pop": ([_vp, _vp, _i64, _i64p, _i64p], ctypes.c_int),
    "ra_router_create": ([_i32, ctypes.POINTER(_vp)], ctypes.c_int),
    "ra_router_destroy": ([_vp], None),
    "ra_router_match": ([_vp, _vp, _i64, _vp], ctypes.c_int),
    "ra_router_insert": ([_vp, _i32, _vp, _i64], ctypes.c_int),
    "ra_router_evict": ([_vp, _i32, _vp, _i64, _i64], ctypes.c_int),
    "ra_router_num_nodes": ([_vp], _i64),
    "ra_router_held_tokens": ([_vp, _i32], _i64),
    "ra_store_kv": ([_vp, _vp, _vp, _i64, _vp, _vp, _i64, _i32, _i32, _vp], ctypes.c_int),
    "ra_extend_attention": ([_vp, _vp, _vp, _i64, _vp, _vp, _i64, _vp, _i64, _i64, _vp, _vp, _vp, _vp,
                             _i32, _i32, _i32, _i32, _i32, ctypes.c_float, _vp, _vp], ctypes.c_int),
    "ra_extend_num_splits": ([_i32, _i32, _i32, _i32, _i32], _i32),
    "ra_extend_workspace_bytes": ([_i64, _i32, _i32, _i32, _i32, _i32, _i32], ctypes.c_size_t),
    "ra_extend_attention_split": ([_vp, _vp, _vp, _i64, _vp, _vp, _i64, _vp, _i64, _i64, _vp, _vp, _vp, _vp,
                                   _i32, _i32, _i32, _i32, _i32, ctypes.c_float, _i32, _vp, ctypes.c_size_t, _vp,
                                   _vp], ctypes.c_int),
    "ra_decode_workspace_bytes": ([_i32, _i32, _i32, _i32, _i32, _i32], ctypes.c_size_t),
    "ra_decode_chunk_len": ([_i32, _i32, _i32, _i32], _i32),
    "ra_decode_attention": ([_vp, _vp, _vp, _i64, _vp, _i64, _i64, _vp, _vp, _i32, _i32, _i32, _i32, _i32,
                             ctypes.c_float, _i32, _vp, ctypes.c_size_t, _vp, _vp], ctypes.c_int),
    "ra_decode_noalloc_max_scratch_bytes": ([], ctypes.c_size_t),
    "ra_decode_attention_noalloc": ([_vp, _vp, _vp, _i64, _vp, _i64, _i64, _vp, _vp, _i32, _i32, _i32, _i32, _i32,
                                     ctypes.c_float, _i32, _vp, _vp], ctypes.c_int),
    "ra_decode_share_plan": ([_vp, _i64, _i64, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _i64, _i64p],
                             ctypes.c_int),
    "ra_decode_shared_workspace_bytes": ([_i32, _i32, _i32], ctypes.c_size_t),
    "ra_decode_attention_shared": ([_vp, _vp, _vp, _i64, _vp, _i64, _i64, _i32, _i32, _i32, _i32, ctypes.c_float,
                                    _vp, _i64, _i32, _i32, _i32, _i32, _vp, ctypes.c_size_t, _vp, _vp], ctypes.c_int),
    "ra_mixed_attention_shared": ([_vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp, _i32, _vp, _i64,
                                   _i32, _i32, _i32, _i32, _vp, ctypes.c_size_t, _vp, _vp, _vp, _i64, _vp, _i64,
                                   _i64, _i32, _i32, _i32, ctypes.c_float, _vp], ctypes.c_int),
    "ra_check_batch": ([_vp, _i64, _i64, _i64, _vp, _i32, _vp, _vp, _vp, _i64, _i32, _vp, _i32, _vp], ctypes.c_int),
    "ra_set_debug_checks": ([_i32], ctypes.c_int),
    "ra_mixed_attention": ([_vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _i32, _i32, _vp,
                            _vp, _vp, _vp, _i32, _i32, _i32, _vp, ctypes.c_size_t, _vp,
                            _vp, _vp, _i64, _vp, _i64, _i64, _i32, _i32, _i32, ctypes.c_float, _vp], ctypes.c_int),
}
for _name, (_args, _res) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res

EXPORTED = tuple(_SIGS)


class RadixAttnError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class OutOfSlots(RadixAttnError):
    pass


def _check(code: int) -> None:
    if code != RA_OK:
        msg = _lib.ra_last_error().decode()
        raise (OutOfSlots if code == RA_ENOMEM else RadixAttnError)(code, msg)


def _np_i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


# ---------------------------------------------------------------------------
# Host radix cache
# ---------------------------------------------------------------------------

class RadixCache:
    """The native radix tree + slot pool (one handle, one scheduler thread)."""

    def __init__(self, pool_slots: int, free_order=None):
        h = _vp()
        order = None if free_order is None else _np_i32(free_order)
        if order is not None and order.shape[0] != pool_slots:
            raise ValueError("free_order must have pool_slots entries")
        _check(_lib.ra_cache_create(pool_slots, None if order is None else order.ctypes.data, ctypes.byref(h)))
        self._h = h
        self.pool_slots = pool_slots

    def __del__(self):
        h = getattr(self, "_h", None)
        lib = _lib  # None once the interpreter is tearing the module down
        if h and lib is not None:
            lib.ra_cache_destroy(h)
            self._h = None

    def match_prefix(self, tokens):
        t = _np_i32(tokens)
        slots = np.empty(t.shape[0], dtype=np.int32)
        n, node = _i64(), _i64()
        _check(_lib.ra_match_prefix(self._h, t.ctypes.data, t.shape[0], slots.ctypes.data,
                                    ctypes.byref(n), ctypes.byref(node)))
        return node.value, n.value, slots[: n.value]

    def inc_ref(self, node: int) -> int:
        d = _i64()
        _check(_lib.ra_inc_ref(self._h, node, ctypes.byref(d)))
        return d.value

    def dec_ref(self, node: int) -> int:
        d = _i64()
        _check(_lib.ra_dec_ref(self._h, node, ctypes.byref(d)))
        return d.value

    def alloc(self, n: int) -> np.ndarray:
        out = np.empty(n, dtype=np.int32)
        _check(_lib.ra_alloc_slots(self._h, n, out.ctypes.data))
        return out

    def free_slots(self, slots) -> None:
        s = _np_i32(slots)
        _check(_lib.ra_free_slots(self._h, s.ctypes.data, s.shape[0]))

    def insert(self, tokens, slots):
        t, s = _np_i32(tokens), _np_i32(slots)
        if t.shape != s.shape:
            raise ValueError("tokens and slots differ in length")
        cached, node = _i64(), _i64()
        _check(_lib.ra_insert(self._h, t.ctypes.data, s.ctypes.data, t.shape[0], ctypes.byref(cached),
                              ctypes.byref(node)))
        return cached.value, node.value

    def evict(self, n_tokens: int) -> int:
        f = _i64()
        _check(_lib.ra_evict(self._h, n_tokens, ctypes.byref(f)))
        return f.value

    def evictable_size(self) -> int:
        return _lib.ra_evictable_size(self._h)

    def available_size(self) -> int:
        return _lib.ra_available_size(self._h)

    def cached_tokens(self) -> int:
        return _lib.ra_cached_tokens(self._h)

    def num_nodes(self) -> int:
        return _lib.ra_num_nodes(self._h)

    def log_evictions(self, enable: bool = True) -> None:
        """Start (or stop and clear) the eviction log."""
        _check(_lib.ra_cache_log_evictions(self._h, 1 if enable else 0))

    def pop_eviction(self):
        """Oldest logged eviction as (root-to-leaf path tokens, evicted suffix
        length), or None when the log is empty."""
        n, k = _i64(), _i64()
        # size probe: an empty log reports -1; otherwise EINVAL with the size
        _lib.ra_eviction_log_pop(self._h, None, 0, ctypes.byref(n), ctypes.byref(k))
        if n.value < 0:
            return None
        buf = np.empty(max(n.value, 1), dtype=np.int32)
        _check(_lib.ra_eviction_log_pop(self._h, buf.ctypes.data, buf.shape[0], ctypes.byref(n), ctypes.byref(k)))
        return buf[: n.value], k.value

    def snapshot(self) -> dict:
        """Same canonical form as the oracle's RadixCache.snapshot()."""
        n = _i64()
        _check(_lib.ra_snapshot(self._h, None, 0, ctypes.byref(n)))
        buf = np.empty(n.value, dtype=np.int64)
        _check(_lib.ra_snapshot(self._h, buf.ctypes.data, n.value, ctypes.byref(n)))
        clock, n_nodes, n_free = int(buf[0]), int(buf[1]), int(buf[2])
        nodes, i = [], 3
        for _ in range(n_nodes):
            nid, parent, ref, stamp, ln = (int(x) for x in buf[i : i + 5])
            i += 5
            key = tuple(int(x) for x in buf[i : i + ln])
            slots = tuple(int(x) for x in buf[i + ln : i + 2 * ln])
            i += 2 * ln
            nodes.append((nid, parent, ref, stamp, key, slots))
        free = [int(x) for x in buf[i : i + n_free]]
        return {"nodes": nodes, "free": free, "clock": clock}


class Router:
    """The native data-parallel router meta-tree (which workers hold which
    prefixes)."""

    def __init__(self, n_workers: int):
        h = _vp()
        _check(_lib.ra_router_create(n_workers, ctypes.byref(h)))
        self._h = h
        self.n_workers = n_workers

    def __del__(self):
        h = getattr(self, "_h", None)
        lib = _lib
        if h and lib is not None:
            lib.ra_router_destroy(h)
            self._h = None

    def match(self, tokens) -> np.ndarray:
        """Per worker, the longest prefix of tokens it holds (router's view)."""
        t = _np_i32(tokens)
        out = np.zeros(self.n_workers, dtype=np.int64)
        _check(_lib.ra_router_match(self._h, t.ctypes.data, t.shape[0], out.ctypes.data))
        return out

    def insert(self, worker: int, tokens) -> None:
        t = _np_i32(tokens)
        _check(_lib.ra_router_insert(self._h, worker, t.ctypes.data, t.shape[0]))

    def evict(self, worker: int, path, evicted_len: int) -> None:
        t = _np_i32(path)
        _check(_lib.ra_router_evict(self._h, worker, t.ctypes.data, t.shape[0], evicted_len))

    def num_nodes(self) -> int:
        return _lib.ra_router_num_nodes(self._h)

    def held_tokens(self, worker: int) -> int:
        return _lib.ra_router_held_tokens(self._h, worker)


# ---------------------------------------------------------------------------
# Device calls (torch tensors; the current stream unless one is given)
# ---------------------------------------------------------------------------

def _stream(stream):
    import torch

    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t, dtype=None, name="tensor"):
    import torch

    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def ra_store_kv(slots, k_new, v_new, k_pool, v_pool, stream=None) -> None:
    import torch

    n, hkv, d = k_new.shape
    _check(_lib.ra_store_kv(_dev(slots, torch.int32, "slots"), _dev(k_new, torch.bfloat16, "k_new"),
                            _dev(v_new, torch.bfloat16, "v_new"), n, _dev(k_pool, torch.bfloat16, "k_pool"),
                            _dev(v_pool, torch.bfloat16, "v_pool"), k_pool.shape[0], hkv, d, _stream(stream)))


def ra_extend_attention(q, k_new, v_new, k_pool, v_pool, req_to_token, req_pool_idx, prefix_lens, extend_lens,
                        extend_start, max_extend_len: int, scale: float, out=None, stream=None):
    import torch

    total, hq, d = q.shape
    hkv = k_new.shape[1]
    if out is None:
        out = torch.empty_like(q)
    _check(_lib.ra_extend_attention(
        _dev(q, torch.bfloat16, "q"), _dev(k_new, torch.bfloat16, "k_new"), _dev(v_new, torch.bfloat16, "v_new"),
        total, _dev(k_pool, torch.bfloat16, "k_pool"), _dev(v_pool, torch.bfloat16, "v_pool"), k_pool.shape[0],
        _dev(req_to_token, torch.int32, "req_to_token"), req_to_token.shape[0], req_to_token.shape[1],
        _dev(req_pool_idx, torch.int32, "req_pool_idx"), _dev(prefix_lens, torch.int32, "prefix_lens"),
        _dev(extend_lens, torch.int32, "extend_lens"), _dev(extend_start, torch.int32, "extend_start"),
        prefix_lens.shape[0], int(max_extend_len), hq, hkv, d, float(scale), _dev(out, torch.bfloat16, "out"),
        _stream(stream)))
    return out


def ra_extend_num_splits(batch: int, max_extend_len: int, hq: int, hkv: int, num_splits: int = 0) -> int:
    return int(_lib.ra_extend_num_splits(batch, max_extend_len, hq, hkv, num_splits))


def ra_extend_workspace_bytes(total_tokens: int, batch: int, max_extend_len: int, hq: int, hkv: int, d: int,
                              num_splits: int = 0) -> int:
    return int(_lib.ra_extend_workspace_bytes(total_tokens, batch, max_extend_len, hq, hkv, d, num_splits))


def ra_extend_attention_split(q, k_new, v_new, k_pool, v_pool, req_to_token, req_pool_idx, prefix_lens, extend_lens,
                              extend_start, max_extend_len: int, scale: float, num_splits: int = 0, workspace=None,
                              out=None, stream=None):
    import torch

    total, hq, d = q.shape
    hkv = k_new.shape[1]
    batch = prefix_lens.shape[0]
    need = ra_extend_workspace_bytes(total, batch, int(max_extend_len), hq, hkv, d, num_splits)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    if out is None:
        out = torch.empty_like(q)
    ws_ptr = _dev(workspace, None, "workspace") if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib.ra_extend_attention_split(
        _dev(q, torch.bfloat16, "q"), _dev(k_new, torch.bfloat16, "k_new"), _dev(v_new, torch.bfloat16, "v_new"),
        total, _dev(k_pool, torch.bfloat16, "k_pool"), _dev(v_pool, torch.bfloat16, "v_pool"), k_pool.shape[0],
        _dev(req_to_token, torch.int32, "req_to_token"), req_to_token.shape[0], req_to_token.shape[1],
        _dev(req_pool_idx, torch.int32, "req_pool_idx"), _dev(prefix_lens, torch.int32, "prefix_lens"),
        _dev(extend_lens, torch.int32, "extend_lens"), _dev(extend_start, torch.int32, "extend_start"),
        batch, int(max_extend_len), hq, hkv, d, float(scale), int(num_splits), ws_ptr, ws_bytes,
        _dev(out, torch.bfloat16, "out"), _stream(stream)))
    return out


def ra_decode_workspace_bytes(batch: int, hq: int, hkv: int, d: int, max_seq_len: int, num_splits: int = 0) -> int:
    return int(_lib.ra_decode_workspace_bytes(batch, hq, hkv, d, max_seq_len, num_splits))


def ra_decode_chunk_len(batch: int, hkv: int, max_seq_len: int, num_splits: int = 0) -> int:
    return int(_lib.ra_decode_chunk_len(batch, hkv, max_seq_len, num_splits))


def ra_decode_attention(q, k_pool, v_pool, req_to_token, req_pool_idx, seq_lens, max_seq_len: int, scale: float,
                        num_splits: int = 0, workspace=None, out=None, stream=None):
    import torch

    b, hq, d = q.shape
    hkv = k_pool.shape[1]
    need = ra_decode_workspace_bytes(b, hq, hkv, d, max_seq_len, num_splits)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    if out is None:
        out = torch.empty_like(q)
    ws_ptr = _dev(workspace, None, "workspace") if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib.ra_decode_attention(
        _dev(q, torch.bfloat16, "q"), _dev(k_pool, torch.bfloat16, "k_pool"), _dev(v_pool, torch.bfloat16, "v_pool"),
        k_pool.shape[0], _dev(req_to_token, torch.int32, "req_to_token"), req_to_token.shape[0],
        req_to_token.shape[1], _dev(req_pool_idx, torch.int32, "req_pool_idx"),
        _dev(seq_lens, torch.int32, "seq_lens"), b, int(max_seq_len), hq, hkv, d, float(scale), int(num_splits),
        ws_ptr, ws_bytes, _dev(out, torch.bfloat16, "out"), _stream(stream)))
    return out


def ra_decode_noalloc_max_scratch_bytes() -> int:
    return int(_lib.ra_decode_noalloc_max_scratch_bytes())


def ra_decode_attention_noalloc(q, k_pool, v_pool, req_to_token, req_pool_idx, seq_lens, max_seq_len: int,
                                scale: float, out, num_splits: int = 0, stream=None):
    """ra_decode_attention without a workspace: the library's per-device
    scratch holds the split partials.  ``out`` is required (this call
    allocates nothing)."""
    import torch

    b, hq, d = q.shape
    hkv = k_pool.shape[1]
    _check(_lib.ra_decode_attention_noalloc(
        _dev(q, torch.bfloat16, "q"), _dev(k_pool, torch.bfloat16, "k_pool"), _dev(v_pool, torch.bfloat16, "v_pool"),
        k_pool.shape[0], _dev(req_to_token, torch.int32, "req_to_token"), req_to_token.shape[0],
        req_to_token.shape[1], _dev(req_pool_idx, torch.int32, "req_pool_idx"),
        _dev(seq_lens, torch.int32, "seq_lens"), b, int(max_seq_len), hq, hkv, d, float(scale), int(num_splits),
        _dev(out, torch.bfloat16, "out"), _stream(stream)))
    return out


class SharePlan:
    """A shared-prefix decode plan (ra_decode_share_plan) on the host, with
    its header counts."""

    def __init__(self, words: np.ndarray):
        self.words = words
        h = words[:16]
        self.n_items, self.n_member_entries, self.n_parts = int(h[0]), int(h[1]), int(h[2])
        self.batch, self.members_per_item, self.rows_per_kv_head = int(h[3]), int(h[4]), int(h[5])
        self.chunk_len = int(h[6])
        o = 16
        self.items = words[o:o + 8 * self.n_items].reshape(-1, 8)
        o += 8 * self.n_items
        self.members = words[o:o + 2 * self.n_member_entries].reshape(-1, 2)
        o += 2 * self.n_member_entries
        self.part_off = words[o:o + self.batch + 1]


def ra_decode_share_plan(req_to_token, req_pool_idx, seq_lens, members_per_item: int, min_shared: int = 256,
                         chunk_len: int = 0, min_items: int = 0) -> SharePlan:
    """Host plan of a shared-prefix decode batch from host copies (numpy) of
    the slot table, the requests' table rows and their context lengths
    (chunk_len 0: the longest chunk giving at least min_items items)."""
    rtt = _np_i32(req_to_token)
    rpi, sl = _np_i32(req_pool_idx), _np_i32(seq_lens)
    if rtt.ndim != 2:
        raise ValueError("req_to_token must be [rows, stride]")
    n = ctypes.c_int64(0)
    args = (rtt.ctypes.data, rtt.shape[0], rtt.shape[1], rpi.ctypes.data, sl.ctypes.data, rpi.shape[0],
            int(members_per_item), int(min_shared), int(chunk_len), int(min_items))
    _check(_lib.ra_decode_share_plan(*args, None, 0, ctypes.byref(n)))
    words = np.zeros(n.value, dtype=np.int32)
    _check(_lib.ra_decode_share_plan(*args, words.ctypes.data, words.shape[0], ctypes.byref(n)))
    return SharePlan(words)


def ra_decode_shared_workspace_bytes(n_parts: int, hq: int, d: int) -> int:
    return int(_lib.ra_decode_shared_workspace_bytes(n_parts, hq, d))


def ra_decode_attention_shared(q, k_pool, v_pool, req_to_token, plan: SharePlan, plan_dev, scale: float,
                               workspace=None, out=None, stream=None):
    """Decode attention over a shared-prefix plan; ``plan_dev`` is the plan's
    words in device memory (int32)."""
    import torch

    b, hq, d = q.shape
    hkv = k_pool.shape[1]
    need = ra_decode_shared_workspace_bytes(plan.n_parts, hq, d)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    if out is None:
        out = torch.empty_like(q)
    ws_ptr = _dev(workspace, None, "workspace") if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib.ra_decode_attention_shared(
        _dev(q, torch.bfloat16, "q"), _dev(k_pool, torch.bfloat16, "k_pool"), _dev(v_pool, torch.bfloat16, "v_pool"),
        k_pool.shape[0], _dev(req_to_token, torch.int32, "req_to_token"), req_to_token.shape[0],
        req_to_token.shape[1], b, hq, hkv, d, float(scale), _dev(plan_dev, torch.int32, "plan"),
        plan_dev.numel(), plan.n_items, plan.n_member_entries, plan.n_parts, plan.members_per_item, ws_ptr,
        ws_bytes, _dev(out, torch.bfloat16, "out"), _stream(stream)))
    return out


def ra_mixed_attention_shared(q_ext, k_new, v_new, req_pool_idx_ext, prefix_lens, extend_lens, extend_start,
                              max_extend_len: int, q_dec, plan: SharePlan, plan_dev, k_pool, v_pool, req_to_token,
                              scale: float, workspace=None, out_ext=None, out_dec=None, stream=None):
    """ra_mixed_attention with the decode half from a shared-prefix plan."""
    import torch

    total, hq, d = q_ext.shape
    hkv = k_pool.shape[1]
    n_dec = q_dec.shape[0]
    need = ra_decode_shared_workspace_bytes(plan.n_parts, hq, d)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q_dec.device)
    if out_ext is None:
        out_ext = torch.empty_like(q_ext)
    if out_dec is None:
        out_dec = torch.empty_like(q_dec)
    ws_ptr = _dev(workspace, None, "workspace") if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib.ra_mixed_attention_shared(
        _dev(q_ext, torch.bfloat16, "q_ext"), _dev(k_new, torch.bfloat16, "k_new"),
        _dev(v_new, torch.bfloat16, "v_new"), total, _dev(req_pool_idx_ext, torch.int32, "req_pool_idx_ext"),
        _dev(prefix_lens, torch.int32, "prefix_lens"), _dev(extend_lens, torch.int32, "extend_lens"),
        _dev(extend_start, torch.int32, "extend_start"), prefix_lens.shape[0], int(max_extend_len),
        _dev(out_ext, torch.bfloat16, "out_ext"), _dev(q_dec, torch.bfloat16, "q_dec"), n_dec,
        _dev(plan_dev, torch.int32, "plan"), plan_dev.numel(), plan.n_items, plan.n_member_entries, plan.n_parts,
        plan.members_per_item, ws_ptr, ws_bytes, _dev(out_dec, torch.bfloat16, "out_dec"),
        _dev(k_pool, torch.bfloat16, "k_pool"), _dev(v_pool, torch.bfloat16, "v_pool"), k_pool.shape[0],
        _dev(req_to_token, torch.int32, "req_to_token"), req_to_token.shape[0], req_to_token.shape[1], hq, hkv, d,
        float(scale), _stream(stream)))
    return out_ext, out_dec


def ra_check_batch(req_to_token, req_pool_idx, pool_slots: int, prefix_lens=None, extend_lens=None,
                   extend_start=None, total_tokens: int = 0, max_extend_len: int = 0, seq_lens=None,
                   max_seq_len: int = 0, stream=None) -> None:
    """Validates an extend batch (prefix_lens, extend_lens, extend_start) or a
    decode batch (seq_lens) on the device; raises RadixAttnError naming the
    first bad request and field."""
    import torch

    opt = lambda t, n: None if t is None else _dev(t, torch.int32, n)  # noqa: E731
    _check(_lib.ra_check_batch(
        _dev(req_to_token, torch.int32, "req_to_token"), req_to_token.shape[0], req_to_token.shape[1],
        int(pool_slots), _dev(req_pool_idx, torch.int32, "req_pool_idx"), req_pool_idx.shape[0],
        opt(prefix_lens, "prefix_lens"), opt(extend_lens, "extend_lens"), opt(extend_start, "extend_start"),
        int(total_tokens), int(max_extend_len), opt(seq_lens, "seq_lens"), int(max_seq_len), _stream(stream)))


def ra_set_debug_checks(enable: bool) -> None:
    """Library-wide debug switch: every attention call validates its batch
    on the device first (see ra_check_batch)."""
    _check(_lib.ra_set_debug_checks(1 if enable else 0))


def ra_mixed_attention(q_ext, k_new, v_new, req_pool_idx_ext, prefix_lens, extend_lens, extend_start,
                       max_extend_len: int, q_dec, req_pool_idx_dec, seq_lens, max_seq_len: int, k_pool, v_pool,
                       req_to_token, scale: float, num_splits: int = 0, workspace=None, out_ext=None, out_dec=None,
                       stream=None):
    """One continuous batch: extend rows and decode rows over the same pool and
    table; extend runs on the current stream, decode on the library's
    companion stream, joined before the call's work completes on `stream`."""
    import torch

    total, hq, d = q_ext.shape
    hkv = k_pool.shape[1]
    n_ext, n_dec = prefix_lens.shape[0], q_dec.shape[0]
    need = ra_decode_workspace_bytes(n_dec, hq, hkv, d, max_seq_len, num_splits)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q_dec.device)
    if out_ext is None:
        out_ext = torch.empty_like(q_ext)
    if out_dec is None:
        out_dec = torch.empty_like(q_dec)
    ws_ptr = _dev(workspace, None, "workspace") if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib.ra_mixed_attention(
        _dev(q_ext, torch.bfloat16, "q_ext"), _dev(k_new, torch.bfloat16, "k_new"),
        _dev(v_new, torch.bfloat16, "v_new"), total, _dev(req_pool_idx_ext, torch.int32, "req_pool_idx_ext"),
        _dev(prefix_lens, torch.int32, "prefix_lens"), _dev(extend_lens, torch.int32, "extend_lens"),
        _dev(extend_start, torch.int32, "extend_start"), n_ext, int(max_extend_len),
        _dev(out_ext, torch.bfloat16, "out_ext"), _dev(q_dec, torch.bfloat16, "q_dec"),
        _dev(req_pool_idx_dec, torch.int32, "req_pool_idx_dec"), _dev(seq_lens, torch.int32, "seq_lens"), n_dec,
        int(max_seq_len), int(num_splits), ws_ptr, ws_bytes, _dev(out_dec, torch.bfloat16, "out_dec"),
        _dev(k_pool, torch.bfloat16, "k_pool"), _dev(v_pool, torch.bfloat16, "v_pool"), k_pool.shape[0],
        _dev(req_to_token, torch.int32, "req_to_token"), req_to_token.shape[0], req_to_token.shape[1], hq, hkv, d,
        float(scale), _stream(stream)))
    return out_ext, out_dec
