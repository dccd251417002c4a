"""Drives a seeded workload through the GPU path (tests, smoke and bench).

The host side uses the package's Scheduler (native radix cache) to build slot
tables; the KV pool's cached positions are filled by the GPU value generator
from each position's prefix hash; new tokens' Q/K/V come from the same
generator and are stored with ``ra_store_kv``.  Nothing here computes
attention: outputs come from the package's kernels.  This module imports the
package and is never imported by the oracle.
"""
from __future__ import annotations

import sys
import time
from dataclasses import dataclass

import numpy as np
import torch

import paper_2312_07104_amd as pa
from paper_2312_07104_amd.runtime import BatchPlan, Scheduler, build_table
from . import contentgen as cg
from . import gpu_gen


def log(*a):
    print(*a, file=sys.stderr, flush=True)


@dataclass
class PhaseInputs:
    plan: BatchPlan
    n_ext: int
    n_dec: int
    hashes: list            # per request, uint64 prefix hashes of its sequence
    table: torch.Tensor     # req_to_token [R, stride] int32
    rpi: torch.Tensor       # req_pool_idx [R] int32 (extends first, then decodes)
    prefix_lens: torch.Tensor
    extend_lens: torch.Tensor
    extend_start: torch.Tensor
    seq_lens: torch.Tensor
    max_extend_len: int
    max_seq_len: int
    total_ext: int
    q_ext: torch.Tensor      # [sum E, Hq, D]
    q_dec: torch.Tensor      # [B_dec, Hq, D]
    k_new: torch.Tensor      # [sum E + B_dec, Hkv, D]
    v_new: torch.Tensor
    new_slots: torch.Tensor  # [sum E + B_dec] int32
    ext_meta: list           # (tokens, P, E, start row)
    dec_meta: list           # (tokens, L)
    table_host: np.ndarray   # host copies of table and rpi (the scheduler builds them on the host)
    rpi_host: np.ndarray


class ScenarioRun:
    def __init__(self, sc, device: str = "cuda", history_limit: int | None = None, row_perm_seed: int = 7,
                 pool=None):
        self.sc = sc
        self.device = device
        self.sched = Scheduler(sc.pool_slots, sc.free_order())
        n_hist = sc.history_len if history_limit is None else min(history_limit, sc.history_len)
        t0 = time.perf_counter()
        for i in range(n_hist):
            self.sched.finish_request(sc.history(i))
        self.history_seconds = time.perf_counter() - t0
        self.history_ops = self.sched.ops
        self.row_perm_seed = row_perm_seed
        if pool is None:
            shape = (sc.pool_slots, sc.hkv, sc.d)
            self.k_pool = torch.empty(shape, dtype=torch.bfloat16, device=device)
            self.v_pool = torch.empty(shape, dtype=torch.bfloat16, device=device)
        else:
            self.k_pool, self.v_pool = pool
        self.filled = np.zeros(sc.pool_slots, dtype=bool)

    # -- inputs --------------------------------------------------------------
    def prepare(self, idx: int) -> PhaseInputs:
        sc, dev = self.sc, self.device
        ph = sc.phases[idx]
        ext = [(r.tokens, r.prefix_len, r.extend_len) for r in ph.extend]
        dec = [(r.tokens, r.seq_len) for r in ph.decode]
        t0 = time.perf_counter()
        plan = self.sched.plan_batch(ext, dec)
        self.plan_seconds = time.perf_counter() - t0
        seqs = [np.asarray(t)[: p + e] for t, p, e in ext] + [np.asarray(t)[:l] for t, l in dec]
        hashes = [cg.prefix_hashes(s, sc.seed) for s in seqs]

        # cached context positions not yet holding their values
        fs, fh = [], []
        for row, h, c in zip(plan.rows, hashes, plan.ctx_lens):
            s = row[:c]
            need = ~self.filled[s]
            fs.append(s[need])
            fh.append(h[:c][need])
        if fs:
            s_all = np.concatenate(fs)
            h_all = np.concatenate(fh)
            s_u, first = np.unique(s_all, return_index=True)
            if s_u.size:
                gpu_gen.fill(self.k_pool, h_all[first], cg.STREAM_K, rows=s_u)
                gpu_gen.fill(self.v_pool, h_all[first], cg.STREAM_V, rows=s_u)
                self.filled[s_u] = True

        n_ext, n_dec = len(ext), len(dec)
        ext_h = [hashes[i][p: p + e] for i, (t, p, e) in enumerate(ext)]
        dec_h = [hashes[n_ext + i][l - 1: l] for i, (t, l) in enumerate(dec)]
        qh_ext = np.concatenate(ext_h) if ext_h else np.zeros(0, np.uint64)
        qh_dec = np.concatenate(dec_h) if dec_h else np.zeros(0, np.uint64)
        new_h = np.concatenate([qh_ext, qh_dec])
        total_ext = int(qh_ext.shape[0])
        hq, hkv, d = sc.hq, sc.hkv, sc.d
        q_ext = torch.empty((max(total_ext, 1), hq, d), dtype=torch.bfloat16, device=dev)[:total_ext]
        q_dec = torch.empty((max(n_dec, 1), hq, d), dtype=torch.bfloat16, device=dev)[:n_dec]
        k_new = torch.empty((max(new_h.shape[0], 1), hkv, d), dtype=torch.bfloat16, device=dev)[: new_h.shape[0]]
        v_new = torch.empty_like(k_new)
        if total_ext:
            gpu_gen.fill(q_ext, qh_ext, cg.STREAM_Q, scale_pow2=sc.q_scale_pow2)
        if n_dec:
            gpu_gen.fill(q_dec, qh_dec, cg.STREAM_Q, scale_pow2=sc.q_scale_pow2)
        if new_h.shape[0]:
            gpu_gen.fill(k_new, new_h, cg.STREAM_K)
            gpu_gen.fill(v_new, new_h, cg.STREAM_V)
        new_slots = np.concatenate(
            [plan.rows[i][p: p + e] for i, (t, p, e) in enumerate(ext)]
            + [plan.rows[n_ext + i][l - 1: l] for i, (t, l) in enumerate(dec)]
        ).astype(np.int32) if (ext or dec) else np.zeros(0, np.int32)

        rng = np.random.default_rng(self.row_perm_seed)
        order = rng.permutation(n_ext + n_dec).astype(np.int32)
        table, rpi = build_table(plan.rows, row_order=order)
        starts = np.cumsum([0] + [e for _, _, e in ext])[:-1] if ext else np.zeros(0, np.int64)
        ext_meta = [(t, p, e, int(s)) for (t, p, e), s in zip(ext, starts)]

        def dt(a):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

        return PhaseInputs(
            plan=plan, n_ext=n_ext, n_dec=n_dec, hashes=hashes, table=dt(table), rpi=dt(rpi),
            prefix_lens=dt([p for _, p, _ in ext]), extend_lens=dt([e for _, _, e in ext]),
            extend_start=dt(starts), seq_lens=dt([l for _, l in dec]),
            max_extend_len=max([e for _, _, e in ext], default=0), max_seq_len=max([l for _, l in dec], default=0),
            total_ext=total_ext, q_ext=q_ext, q_dec=q_dec, k_new=k_new, v_new=v_new,
            new_slots=dt(new_slots), ext_meta=ext_meta, dec_meta=dec, table_host=np.ascontiguousarray(table, dtype=np.int32),
            rpi_host=np.ascontiguousarray(rpi, dtype=np.int32))

    # -- the hot path ----------------------------------------------------------
    def store(self, inp: PhaseInputs) -> None:
        if inp.new_slots.shape[0]:
            pa.ra_store_kv(inp.new_slots, inp.k_new, inp.v_new, self.k_pool, self.v_pool)
            self.filled[inp.new_slots.cpu().numpy()] = True

    def extend(self, inp: PhaseInputs, out=None, num_splits: int | None = None, workspace=None):
        """ra_extend_attention, or ra_extend_attention_split when
        ``num_splits`` is given (0: the library picks the key splits)."""
        if inp.n_ext == 0:
            return None
        args = (inp.q_ext, inp.k_new[: inp.total_ext], inp.v_new[: inp.total_ext], self.k_pool, self.v_pool,
                inp.table, inp.rpi[: inp.n_ext], inp.prefix_lens, inp.extend_lens, inp.extend_start,
                inp.max_extend_len, self.sc.scale)
        if num_splits is None:
            return pa.ra_extend_attention(*args, out=out)
        return pa.ra_extend_attention_split(*args, num_splits=num_splits, workspace=workspace, out=out)

    def extend_workspace_bytes(self, inp: PhaseInputs, num_splits: int = 0) -> int:
        if inp.n_ext == 0:
            return 0
        return pa.ra_extend_workspace_bytes(inp.total_ext, inp.n_ext, inp.max_extend_len, self.sc.hq, self.sc.hkv,
                                            self.sc.d, num_splits)

    def decode(self, inp: PhaseInputs, num_splits: int = 0, workspace=None, out=None):
        if inp.n_dec == 0:
            return None
        return pa.ra_decode_attention(
            inp.q_dec, self.k_pool, self.v_pool, inp.table, inp.rpi[inp.n_ext:], inp.seq_lens, inp.max_seq_len,
            self.sc.scale, num_splits=num_splits, workspace=workspace, out=out)

    def share_plan(self, inp: PhaseInputs, members_per_item: int | None = None, min_shared: int = 256,
                   chunk_len: int = 0, min_items: int | None = None):
        """Host plan of the decode half for ra_decode_attention_shared (from
        host copies of the table, the decode requests' rows and lengths) and
        its words in device memory.  Defaults: members_per_item fills two
        16-column MFMA blocks with query heads (32 / G requests, 1 .. 16);
        chunk_len 0 with min_items = one wave per SIMD over the kv heads."""
        grp = self.sc.hq // self.sc.hkv
        if members_per_item is None:
            members_per_item = max(1, min(16, 32 // grp))
        if min_items is None:
            cus = torch.cuda.get_device_properties(0).multi_processor_count if torch.cuda.is_available() else 256
            min_items = -(-4 * cus // self.sc.hkv)
        t0 = time.perf_counter()
        lens = np.array([l for _, l in inp.dec_meta], dtype=np.int32)
        plan = pa.ra_decode_share_plan(inp.table_host, inp.rpi_host[inp.n_ext:], lens, members_per_item, min_shared,
                                       chunk_len, min_items)
        self.share_plan_seconds = time.perf_counter() - t0
        return plan, torch.from_numpy(plan.words).to(self.device)

    def decode_shared(self, inp: PhaseInputs, plan, plan_dev, workspace=None, out=None):
        if inp.n_dec == 0:
            return None
        return pa.ra_decode_attention_shared(inp.q_dec, self.k_pool, self.v_pool, inp.table, plan, plan_dev,
                                             self.sc.scale, workspace=workspace, out=out)

    def mixed_shared(self, inp: PhaseInputs, plan, plan_dev, workspace=None, out_ext=None, out_dec=None,
                     ext_splits: int | None = None, ext_workspace=None):
        """Both halves in one ra_mixed_attention_shared call (the decode half
        from a shared-prefix plan).  A batch without extends or decodes goes
        to the one entry point it needs."""
        if inp.n_dec == 0:
            return self.extend(inp, out=out_ext, num_splits=ext_splits, workspace=ext_workspace), None
        if inp.n_ext == 0:
            return None, self.decode_shared(inp, plan, plan_dev, workspace=workspace, out=out_dec)
        return pa.ra_mixed_attention_shared(
            inp.q_ext, inp.k_new[: inp.total_ext], inp.v_new[: inp.total_ext], inp.rpi[: inp.n_ext],
            inp.prefix_lens, inp.extend_lens, inp.extend_start, inp.max_extend_len, inp.q_dec, plan, plan_dev,
            self.k_pool, self.v_pool, inp.table, self.sc.scale, workspace=workspace, out_ext=out_ext,
            out_dec=out_dec)

    def mixed(self, inp: PhaseInputs, num_splits: int = 0, workspace=None, out_ext=None, out_dec=None,
              ext_splits: int | None = None, ext_workspace=None):
        """Both halves of the batch in one ra_mixed_attention call.  A batch
        without decodes goes to the extend entry point, the split one when
        ``ext_splits`` is given."""
        if inp.n_ext == 0 or inp.n_dec == 0:
            return (self.extend(inp, out=out_ext, num_splits=ext_splits, workspace=ext_workspace),
                    self.decode(inp, num_splits, workspace, out_dec))
        return pa.ra_mixed_attention(
            inp.q_ext, inp.k_new[: inp.total_ext], inp.v_new[: inp.total_ext], inp.rpi[: inp.n_ext],
            inp.prefix_lens, inp.extend_lens, inp.extend_start, inp.max_extend_len, inp.q_dec,
            inp.rpi[inp.n_ext:], inp.seq_lens, inp.max_seq_len, self.k_pool, self.v_pool, inp.table, self.sc.scale,
            num_splits=num_splits, workspace=workspace, out_ext=out_ext, out_dec=out_dec)

    def finish(self, idx: int, inp: PhaseInputs) -> None:
        ph = self.sc.phases[idx]
        ext = [(r.tokens, r.prefix_len, r.extend_len) for r in ph.extend]
        dec = [(r.tokens, r.seq_len) for r in ph.decode]
        self.sched.finish_batch(ext, dec, inp.plan)
