"""Benchmark of the RadixAttention hot path on one MI355X.

One step = one pass of the whole hot path over one continuous batch: store the
batch's new tokens' K/V into their pool slots, extend attention for the
extend requests, decode attention (partial pass + combine) for the decode
requests.  The slot tables come from the native radix cache after replaying
the workload's request history (host time reported separately).

Default workload: the continuous-batching mix with 70B-like heads (64 query
heads, 8 kv heads, head dim 128): 32 extend requests (cached prefix
U[1024, 8192], extend U[256, 2048]) and 512 decode requests (context
U[1024, 16384]) over a 4,194,304-slot pool, tables built by ~100k tree calls.

Prints one JSON line.  Before anything is timed, untimed steps run for
--clock-warmup seconds (the GPU's clocks ramp up over the first tens of
milliseconds of sustained load), then the W warm-up steps.  The headline loop
runs the steps back to back (the
mixed call overlaps extend and decode on two streams).  A second loop runs the
same work one kernel at a time, each step after a 1 GiB write that evicts L2
and the Infinity Cache (cold caches), with HIP events recorded on the stream
the kernels run on; its per-kernel durations give the rooflines.  HBM traffic
per launch comes from rocprofv3 FETCH_SIZE / WRITE_SIZE passes stored in
profiles/traffic.json, and is reported only while the kernel sources still
hash to the values recorded there.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
FLUSH_BYTES = 1 << 30
CSRC = os.path.join(ROOT, "paper_2312_07104_amd", "csrc")
# sources whose code a kernel's launch runs (traffic figures are tied to them)
KERNEL_SOURCES = {
    "extend": ["extend.hip", "lds_dma.h", "device_common.h"],
    "decode": ["decode.hip", "decode_shared.hip", "lds_dma.h", "device_common.h"],
}


def sources_sha256(kernel):
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(kernel, workload, decode_path=None):
    """HBM bytes per step of a kernel (all its launches in the step: the
    partial pass and its combine) from the committed counter summary, or None
    when it is missing, was taken on different kernel sources or, for decode,
    on the other decode path."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh).get(f"{kernel}/{workload}")
    except (OSError, ValueError):
        return None
    if not rec or rec.get("sources_sha256") != sources_sha256(kernel):
        return None
    if kernel == "decode" and rec.get("decode_path") != decode_path:
        return None
    return rec.get("hbm_bytes_per_launch")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_work(sc, inp):
    """Algorithmic flops of extend and bytes of decode for one step.

    Extend: 4*D flops (QK^T and PV) per unmasked (query head, query, key)
    triple: Hq * sum_r (E_r * P_r + E_r (E_r + 1) / 2).
    Decode: each request reads K and V rows of its kv heads for all L_r
    positions (2 * Hkv * D * 2 bytes), its slot index (4 bytes), its query
    and writes its output (2 * Hq * D * 2 bytes).
    """
    hq, hkv, d = sc.hq, sc.hkv, sc.d
    pairs = sum(e * p + e * (e + 1) // 2 for _, p, e, _ in inp.ext_meta)
    ext_flops = 4.0 * d * hq * pairs
    ext_bytes = sum((p + e) * (2 * hkv * d * 2) + p * 4 + e * (2 * hq * d * 2) for _, p, e, _ in inp.ext_meta)
    # distinct K/V rows over the extend contexts (a position is named by the
    # hash of its prefix, so requests sharing a prefix share its rows)
    from workload import contentgen as cg
    seen = set()
    for h in cg.prefix_hashes_batch([toks[:p + e] for toks, p, e, _ in inp.ext_meta], sc.seed) if inp.ext_meta else []:
        seen.update(h.tolist())
    ext_unique_bytes = len(seen) * (2 * hkv * d * 2) + sum(e * (2 * hq * d * 2) for _, _, e, _ in inp.ext_meta)
    sum_l = sum(l for _, l in inp.dec_meta)
    dec_bytes = sum_l * (2 * hkv * d * 2 + 4) + inp.n_dec * 2 * hq * d * 2
    dec_flops = 4.0 * d * hq * sum_l
    attended = sum(p + e for _, p, e, _ in inp.ext_meta) + sum_l
    return dict(ext_flops=ext_flops, ext_bytes=ext_bytes, ext_unique_bytes=ext_unique_bytes, dec_bytes=dec_bytes, dec_flops=dec_flops,
                attended=attended, sum_l=sum_l, pairs=pairs)


def cpu_baseline(sc, inp, budget_s: float, workers: int):
    """The oracle, timed on the host's cores over a bounded sample of the batch.

    Requests go to a pool of worker processes (spawned, one thread each:
    OpenMP and BLAS limited to one), the shortest extend request first, then
    the decode requests in batch order, every worker kept busy until the time
    budget is spent (running requests finish).  Workers start and import the
    oracle before the timing starts.  Each request regenerates its inputs from
    its own token list and attends in float64; regeneration and attention are
    timed separately inside the workers."""
    from oracle import pool as opool

    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas_threads = None
    tasks, ctx, flops = [], [], []
    if inp.ext_meta:
        toks, p, e, _ = min(inp.ext_meta, key=lambda m: m[2] * (m[1] + m[2]))
        tasks.append(opool.extend_task(toks, p, e, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale))
        ctx.append(p + e)
        flops.append(4.0 * sc.d * sc.hq * (e * p + e * (e + 1) // 2))
    for toks, l in inp.dec_meta:
        tasks.append(opool.decode_task(toks, l, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale))
        ctx.append(l)
        flops.append(4.0 * sc.d * sc.hq * l)
    with opool.OraclePool(workers, threads_per_worker=1) as pool:
        pool.warm()
        done, wall = pool.run_for(tasks, budget_s)
    idx = [i for i, _, _ in done]
    tokens = sum(ctx[i] for i in idx)
    n_ext = sum(1 for i in idx if inp.ext_meta and i == 0)
    regen = sum(tm.get("regen", 0.0) for _, _, tm in done)
    attend = sum(tm.get("attend", 0.0) for _, _, tm in done)
    return {"value": tokens / wall, "unit": "attended KV tokens/s", "cores": workers, "kind": "oracle",
            "processes": workers, "threads_per_process": 1, "affinity_cores": len(os.sched_getaffinity(0)),
            "blas_threads_in_parent": blas_threads,
            "gflops": sum(flops[i] for i in idx) / wall / 1e9,
            "wall_s": wall, "regen_cpu_s": regen, "attend_cpu_s": attend,
            "sample": f"{n_ext} extend + {len(idx) - n_ext} decode requests of the batch ({tokens} context tokens "
                      f"in {wall:.1f} s on {workers} worker processes of one thread each; each request "
                      f"regenerates its inputs from its token list: {regen:.0f} CPU-s regeneration, "
                      f"{attend:.0f} CPU-s float64 attention)"}


def scheduler_report(sc, n: int = 300):
    """Theorem 3.1 on the workload's own request stream: the first n history
    requests as one offline batch, cache = the longest of them, processed in
    longest-shared-prefix-first, submission and random order; computed tokens
    against the sum of the batch's radix-tree edge lengths."""
    from paper_2312_07104_amd.runtime import run_offline

    seqs = [np.asarray(sc.history(i), dtype=np.int32) for i in range(min(n, sc.history_len))]
    if not seqs:
        return None
    root: dict = {}
    edges = 0  # distinct non-empty prefixes = trie nodes below the root
    for s in seqs:
        node = root
        for t in s.tolist():
            nxt = node.get(t)
            if nxt is None:
                nxt = node[t] = {}
                edges += 1
            node = nxt
    pool = max(len(s) for s in seqs)
    out = {"requests": len(seqs), "prefill_tokens": int(sum(len(s) for s in seqs)), "edge_tokens": edges,
           "cache_slots": pool}
    t0 = time.perf_counter()
    for policy in ("lspf", "fcfs", "random"):
        r = run_offline(seqs, pool, policy, seed=1)
        out[policy] = {"computed_tokens": r.computed_tokens, "hit_rate": r.hit_rate}
    out["seconds"] = time.perf_counter() - t0
    return out


def data_parallel_report(sc, n: int = 2000, n_workers: int = 4):
    """Appendix A.4 on the workload's own stream: the first n history requests
    dispatched over n_workers replicas (each with a quarter of a cache sized
    for about a fifth of the stream's tokens) by the router meta-tree, with
    the affinity policy and with cache-blind policies; a single cache of the
    same total size is the bound.  Evictions are committed to the router
    every 50 requests."""
    from paper_2312_07104_amd.runtime import run_data_parallel

    seqs = [np.asarray(sc.history(i), dtype=np.int32) for i in range(min(n, sc.history_len))]
    if not seqs:
        return None
    total = sum(len(x) for x in seqs)
    per_worker = max(max(len(x) for x in seqs), total // (5 * n_workers))
    t0 = time.perf_counter()
    single = run_data_parallel(seqs, 1, n_workers * per_worker, "least_loaded")
    out = {"requests": len(seqs), "prefill_tokens": total, "workers": n_workers, "slots_per_worker": per_worker,
           "commit_every": 50, "single_cache_hit_rate": single.hit_rate}
    for policy in ("affinity", "least_loaded", "round_robin", "random"):
        r = run_data_parallel(seqs, n_workers, per_worker, policy, commit_every=50, seed=1)
        out[policy] = {"hit_rate": r.hit_rate, "imbalance": r.imbalance, "router_nodes": r.router_nodes}
    out["seconds"] = time.perf_counter() - t0
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--clock-warmup", type=float, default=1.0,
                    help="seconds of untimed steps before the W warm-up steps: the GPU's clocks ramp up over "
                         "the first tens of milliseconds of sustained load")
    ap.add_argument("--workload", default="mixed")
    ap.add_argument("--phase", type=int, default=0,
                    help="batch of the workload to time; earlier batches run and finish first (their new tokens "
                         "are stored and their sequences inserted)")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--cpu-workers", type=int, default=max(1, min(16, len(os.sched_getaffinity(0)))),
                    help="oracle worker processes for the CPU baseline (one thread each)")
    ap.add_argument("--no-peaks", action="store_true", help="skip the machine-peak microbenchmarks")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--decode", choices=("shared", "per-request"), default="shared",
                    help="decode half: shared-prefix plan (each shared run of the batch read once per block of "
                         "requests) or one pass per request")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the timed loop, run one device copy of this size (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the path shards by request, "
              f"see the design notes", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2312_07104_amd as pa
    from workload.driver import ScenarioRun
    from workload import scenarios as S

    sc = S.ALL[args.workload]()
    log(f"[bench] workload={sc.name} seed={sc.seed} Hq={sc.hq} Hkv={sc.hkv} D={sc.d} S={sc.pool_slots}")
    run = ScenarioRun(sc)
    log(f"[bench] history: {sc.history_len} requests, {run.history_ops} tree calls, {run.history_seconds:.2f} s")
    for ph in range(args.phase):
        prev = run.prepare(ph)
        run.store(prev)
        run.finish(ph, prev)
    inp = run.prepare(args.phase)
    log(f"[bench] batch planned: {run.plan_seconds * 1e3:.1f} ms host, hit rate {inp.plan.hit_rate:.3f}")
    run.store(inp)  # the first pass writes new tokens' K/V (identical values every step)
    torch.cuda.synchronize()
    work = algorithmic_work(sc, inp)

    stream = torch.cuda.current_stream()
    n_new = inp.new_slots.shape[0]
    ws_bytes = pa.ra_decode_workspace_bytes(inp.n_dec, sc.hq, sc.hkv, sc.d, inp.max_seq_len, 0)
    workspace = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    out_e = torch.empty_like(inp.q_ext) if inp.n_ext else None
    out_d = torch.empty_like(inp.q_dec) if inp.n_dec else None

    ws_t = workspace if ws_bytes else None
    # A batch without decodes takes the extend entry point with key splits
    # (the library picks them; none when the work items already fill the chip).
    ext_ws_bytes = run.extend_workspace_bytes(inp, 0) if inp.n_ext else 0
    ext_ws = torch.empty(ext_ws_bytes, dtype=torch.uint8, device="cuda") if ext_ws_bytes else None
    ext_splits = 0 if inp.n_dec == 0 else None
    ext_ns = pa.ra_extend_num_splits(inp.n_ext, inp.max_extend_len, sc.hq, sc.hkv, 0) if ext_splits == 0 else 1
    log(f"[bench] extend key splits: {ext_ns}")
    # Decode half from a shared-prefix plan, made on the host from the batch's
    # slot rows before the timed region (its host time is reported).
    use_shared = args.decode == "shared" and inp.n_dec > 0
    plan = plan_dev = sh_ws = None
    share = None
    if use_shared:
        plan, plan_dev = run.share_plan(inp)
        sh_need = pa.ra_decode_shared_workspace_bytes(plan.n_parts, sc.hq, sc.d)
        sh_ws = torch.empty(sh_need, dtype=torch.uint8, device="cuda") if sh_need else None
        rows = plan.rows_per_kv_head * sc.hkv
        # bytes the plan's items must move: K and V rows and slot indices of
        # every item, queries, outputs, and each partial written and read once
        plan_bytes = (rows * (2 * sc.d * 2 + 4) + inp.n_dec * 2 * sc.hq * sc.d * 2
                      + 2 * plan.n_parts * sc.hq * (sc.d + 1) * 4)
        share = {"members_per_item": plan.members_per_item, "chunk_len": plan.chunk_len, "items": plan.n_items,
                 "partials": plan.n_parts, "rows_read": rows, "rows_per_request": work["sum_l"] * sc.hkv,
                 "rows_read_fraction": rows / max(work["sum_l"] * sc.hkv, 1), "plan_bytes": plan_bytes,
                 "host_plan_ms": run.share_plan_seconds * 1e3}
        log(f"[bench] shared-prefix decode: {plan.n_items} items, {plan.n_parts} partials, "
            f"{share['rows_read_fraction']:.3f} of the per-request rows, host plan {share['host_plan_ms']:.1f} ms")
    flush_buf = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device="cuda")

    def step():
        """One pass of the hot path: store new K/V, then the mixed batch call."""
        if n_new:
            pa.ra_store_kv(inp.new_slots, inp.k_new, inp.v_new, run.k_pool, run.v_pool)
        if use_shared:
            run.mixed_shared(inp, plan, plan_dev, workspace=sh_ws, out_ext=out_e, out_dec=out_d,
                             ext_splits=ext_splits, ext_workspace=ext_ws)
        else:
            run.mixed(inp, workspace=ws_t, out_ext=out_e, out_dec=out_d, ext_splits=ext_splits,
                      ext_workspace=ext_ws)

    def step_sequential(ev):
        """The same work with each kernel timed alone (for the rooflines)."""
        ev[0].record(stream)
        if n_new:
            pa.ra_store_kv(inp.new_slots, inp.k_new, inp.v_new, run.k_pool, run.v_pool)
        ev[1].record(stream)
        if inp.n_ext:
            run.extend(inp, out=out_e, num_splits=ext_splits, workspace=ext_ws)
        ev[2].record(stream)
        if inp.n_dec:
            if use_shared:
                run.decode_shared(inp, plan, plan_dev, workspace=sh_ws, out=out_d)
            else:
                run.decode(inp, workspace=ws_t, out=out_d)
        ev[3].record(stream)

    clock_steps = 0
    t_cw = time.perf_counter()
    while time.perf_counter() - t_cw < args.clock_warmup:
        step()
        torch.cuda.synchronize()
        clock_steps += 1
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        flush_buf.fill_(i & 0xFF)  # cold L2 / Infinity Cache for the timed kernels
        step_sequential(events[i])
    torch.cuda.synchronize()
    ms_seq = float(np.mean([e[0].elapsed_time(e[3]) for e in events]))
    per_step = {"store_kv": [e[0].elapsed_time(e[1]) for e in events],
                "extend": [e[1].elapsed_time(e[2]) for e in events],
                "decode": [e[2].elapsed_time(e[3]) for e in events]}
    t_store = float(np.mean(per_step["store_kv"]))
    t_ext = float(np.mean(per_step["extend"]))
    t_dec = float(np.mean(per_step["decode"]))

    kernels = {
        "store_kv": {"ms": t_store, "tokens": int(n_new)},
        "extend": {"ms": t_ext, "tflops": work["ext_flops"] / (t_ext * 1e-3) / 1e12,
                   "flops": work["ext_flops"], "gbs": work["ext_bytes"] / (t_ext * 1e-3) / 1e9,
                   "bytes": work["ext_bytes"], "unique_bytes": work["ext_unique_bytes"]} if inp.n_ext else None,
        "decode": {"ms": t_dec, "gbs": work["dec_bytes"] / (t_dec * 1e-3) / 1e9,
                   "bytes": work["dec_bytes"], "path": args.decode} if inp.n_dec else None,
    }

    def extend_roof():
        """Extend is bounded by MFMA when its algorithmic intensity (flops per
        byte of distinct K/V rows, queries and outputs: a prefix shared by
        several requests is fetched once and served from L2 / the Infinity
        Cache) is above the ridge point of the two peaks, by HBM below it
        (short extends over long cached prefixes).  The HBM figure itself is
        the per-request byte count, like decode's."""
        e = kernels["extend"]
        if work["ext_flops"] / max(work["ext_unique_bytes"], 1) >= BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
            return {"kernel": "extend", "bound": "mfma", "achieved": e["tflops"], "peak": BF16_PEAK_TFLOPS,
                    "unit": "TFLOP/s"}
        return {"kernel": "extend", "bound": "hbm", "achieved": e["gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s"}

    if share and kernels["decode"]:
        kernels["decode"]["plan_bytes"] = share["plan_bytes"]
        kernels["decode"]["plan_gbs"] = share["plan_bytes"] / (t_dec * 1e-3) / 1e9

    def decode_roof():
        """Decode is HBM-bound.  The shared-prefix path is priced on the bytes
        its plan must move (each shared run once per block of requests); the
        per-request byte rate, which counts every request's rows, is kept
        beside it as logical_gbs."""
        d = kernels["decode"]
        r = {"kernel": "decode", "bound": "hbm", "achieved": d.get("plan_gbs", d["gbs"]), "peak": HBM_PEAK_GBS,
             "unit": "GB/s"}
        if "plan_gbs" in d:
            r["logical_gbs"] = d["gbs"]
        return r

    # roofline: the kernel that takes longer; roofline_other: the other one
    first, second = (extend_roof, decode_roof) if inp.n_ext and t_ext >= t_dec else (decode_roof, extend_roof)
    roof = first()
    other = second() if (kernels["decode"] if second is decode_roof else kernels["extend"]) else None
    for name, k in kernels.items():
        if k:
            k["ms_median"] = float(np.median(per_step[name]))
            k["ms_min"] = float(np.min(per_step[name]))
    for r in (roof, other):
        if r:
            r["frac"] = r["achieved"] / r["peak"]
            r["traffic"] = measured_traffic(r["kernel"], sc.name, args.decode)
            # HBM bytes the counters saw per launch over the kernel's duration
            if r["traffic"]:
                r["hbm_gbs"] = r["traffic"] / (kernels[r["kernel"]]["ms"] * 1e-3) / 1e9
                r["hbm_frac"] = r["hbm_gbs"] / HBM_PEAK_GBS

    peaks = None
    if not args.no_peaks:
        from workload import peaks as pk

        log("[bench] measuring machine peaks (streaming read, 256-byte gathers, MFMA loops)")
        peaks = pk.measure()
        for r in (roof, other):
            if not r:
                continue
            if r["unit"] == "TFLOP/s":
                r["measured_peak"] = max(peaks["mfma16_bf16_tflops"], peaks["mfma32_bf16_tflops"])
                r["frac_of_measured"] = r["achieved"] / r["measured_peak"]
            else:
                r["measured_peak"] = max(peaks["gather256_gbs"], peaks["gather_kv_gbs"], peaks["hbm_read_gbs"])
                r["frac_of_measured"] = r["achieved"] / r["measured_peak"]
                if r.get("hbm_gbs"):
                    r["hbm_frac_of_measured"] = r["hbm_gbs"] / r["measured_peak"]

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy: {n} bytes read, {n} bytes written")

    value = work["attended"] / (ms_step * 1e-3)
    line = {
        "metric": "attended KV tokens/s (extend + decode step over the radix-cached KV pool)",
        "value": value, "unit": "attended KV tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": sc.name, "phase": args.phase, "hq": sc.hq, "hkv": sc.hkv, "head_dim": sc.d,
                   "pool_slots": sc.pool_slots, "extend_requests": inp.n_ext, "decode_requests": inp.n_dec,
                   "sum_extend_tokens": inp.total_ext, "sum_decode_context": work["sum_l"],
                   "history_requests": sc.history_len, "tree_calls": run.history_ops,
                   "hit_rate": inp.plan.hit_rate, "extend_key_splits": ext_ns if inp.n_ext else None,
                   "decode_path": args.decode if inp.n_dec else None, "decode_share": share,
                   "parallelism": "none (1 GPU)"},
        "clock_warmup": {"seconds": args.clock_warmup, "steps": clock_steps},
        "ms_per_step_sequential_cold": ms_seq,
        "roofline": roof,
        "roofline_other": other,
        "peaks_measured": peaks,
        "kernels": kernels,
        "host_tree": {"calls": run.history_ops, "seconds": run.history_seconds,
                      "calls_per_s": run.history_ops / max(run.history_seconds, 1e-9),
                      "plan_batch_ms": run.plan_seconds * 1e3,
                      "plan_batch_requests": inp.n_ext + inp.n_dec,
                      "plan_ms_per_request": run.plan_seconds * 1e3 / max(inp.n_ext + inp.n_dec, 1)},
    }
    line["scheduler"] = scheduler_report(sc)
    line["data_parallel"] = data_parallel_report(sc)
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on host cores")
        line["cpu_baseline"] = cpu_baseline(sc, inp, args.cpu_budget, args.cpu_workers)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
