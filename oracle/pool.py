"""Runs the oracle's per-request references over a pool of worker processes.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The oracle recomputes every request from scratch and independently of the
others, so a batch's requests can be spread over processes without changing
any request's arithmetic: each task is one call of ``extend_reference`` or
``decode_reference`` with the same arguments it would get in-process.

Workers are started with the ``spawn`` method (a fresh interpreter per
worker, which imports only NumPy, this package and ``workload.contentgen``),
so a parent that has already initialised a GPU never forks its state.  Each
worker limits its own OpenMP and BLAS threads so that the pool does not
oversubscribe the host's cores.
"""
from __future__ import annotations

import concurrent.futures as cf
import multiprocessing as mp
import os
import time

import numpy as np


def _init_worker(threads: int) -> None:
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = str(threads)
    try:
        from threadpoolctl import threadpool_limits

        threadpool_limits(threads)
    except Exception:  # pragma: no cover - threadpoolctl is optional
        pass


def _run_task(task):
    """task = (kind, kwargs); returns (result, {"regen": s, "attend": s})."""
    from . import attention as oa

    kind, kw = task
    tm: dict = {}
    if kind == "decode":
        out = oa.decode_reference(**kw, timings=tm)
    elif kind == "extend":
        out = oa.extend_reference(**kw, timings=tm)
    else:
        raise ValueError(kind)
    return out, tm


def decode_task(tokens, seq_len, seed, hq, hkv, d, scale, q_scale_pow2=0, key_patches=None):
    return ("decode", dict(tokens=np.asarray(tokens), seq_len=int(seq_len), seed=seed, hq=hq, hkv=hkv, d=d,
                           scale=scale, q_scale_pow2=q_scale_pow2, key_patches=key_patches))


def extend_task(tokens, prefix_len, extend_len, seed, hq, hkv, d, scale, q_scale_pow2=0, rows=None,
                key_patches=None):
    return ("extend", dict(tokens=np.asarray(tokens), prefix_len=int(prefix_len), extend_len=int(extend_len),
                           seed=seed, hq=hq, hkv=hkv, d=d, scale=scale, q_scale_pow2=q_scale_pow2,
                           rows=None if rows is None else np.asarray(rows), key_patches=key_patches))


def default_workers() -> int:
    return max(1, min(16, len(os.sched_getaffinity(0))))


class OraclePool:
    """A spawn-started process pool for oracle tasks (use as a context manager).

    A worker that cannot start (for instance when the parent's main module
    cannot be re-imported) breaks the pool, and every pending task then
    raises instead of waiting forever.
    """

    def __init__(self, workers: int | None = None, threads_per_worker: int = 1):
        self.workers = workers or default_workers()
        self.threads_per_worker = threads_per_worker
        self._ex = None

    def __enter__(self):
        self._ex = cf.ProcessPoolExecutor(self.workers, mp_context=mp.get_context("spawn"),
                                          initializer=_init_worker, initargs=(self.threads_per_worker,))
        return self

    def __exit__(self, *exc):
        self._ex.shutdown(wait=True, cancel_futures=True)
        self._ex = None

    def imap(self, tasks):
        """Yields (index, result, {"regen": s, "attend": s}) as tasks finish
        (in any order)."""
        futs = {self._ex.submit(_run_task, t): i for i, t in enumerate(tasks)}
        for f in cf.as_completed(futs):
            out, tm = f.result()
            yield futs[f], out, tm

    def warm(self) -> None:
        """Starts every worker and imports the oracle in it (a tiny task per
        worker), so that later timings exclude interpreter start-up."""
        tiny = decode_task(np.arange(4, dtype=np.int32), 4, 1, 1, 1, 16, 0.25)
        list(self.imap([tiny] * (2 * self.workers)))

    def run_for(self, tasks, seconds: float):
        """Runs tasks in order with every worker busy and stops submitting
        new ones once ``seconds`` have passed (running ones finish).
        Returns ([(index, result, timings)], wall seconds)."""
        t0 = time.perf_counter()
        it = iter(enumerate(tasks))
        pending = {}

        def submit() -> None:
            nxt = next(it, None)
            if nxt is not None:
                pending[self._ex.submit(_run_task, nxt[1])] = nxt[0]

        for _ in range(self.workers):
            submit()
        done = []
        while pending:
            fin, _ = cf.wait(pending, return_when=cf.FIRST_COMPLETED)
            for f in fin:
                i = pending.pop(f)
                out, tm = f.result()
                done.append((i, out, tm))
                if time.perf_counter() - t0 < seconds:
                    submit()
        return done, time.perf_counter() - t0

    def map(self, tasks) -> list:
        res = [None] * len(tasks)
        for i, out, _ in self.imap(tasks):
            res[i] = out
        return res
