"""GPU-side helpers of the parity tests: needle planting, the table -> pool
content check and oracle comparisons over a process pool.

The workload driver (``workload.driver``) builds the inputs and calls the
package's kernels; expected values come from the oracle.  Nothing here
computes attention.  Tolerances and needle arithmetic live in ``tests.gate``.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

from oracle import pool as opool
from tests.gate import MAX_ABS, MEAN_ABS, REL_RMS, assert_close, errors, needle_key  # noqa: F401
from workload import contentgen as cg
from workload import gpu_gen
from workload.driver import PhaseInputs, ScenarioRun, log  # noqa: F401  (re-exported for the tests)


def make_scenario(name, hq, hkv, d, pool, extend=(), decode=(), seed=77, q_pow2=0):
    """A one-batch scenario of private token runs: extend requests (P, E) and
    decode requests of context L, no history."""
    from workload import scenarios as S

    ext = [S.ExtendReq(cg.run_tokens(seed * 1000 + i, p + e, S.VOCAB), p, e) for i, (p, e) in enumerate(extend)]
    dec = [S.DecodeReq(cg.run_tokens(seed * 1000 + 500 + i, l, S.VOCAB), l) for i, l in enumerate(decode)]
    sc = S.Scenario(name, seed, hq, hkv, d, pool, 0, lambda i: None, [S.Phase(extend=ext, decode=dec)])
    sc.q_scale_pow2 = q_pow2
    return sc


@dataclass
class Needle:
    """A planted key: request ``req`` of kind "ext" (query = new token ``row``,
    position P + row) or "dec" (query at L - 1); query head ``head``; key
    position ``pos`` (<= the query's position)."""
    kind: str
    req: int
    head: int
    pos: int
    row: int = 0
    share: float = 0.5


def _req_view(inp: PhaseInputs, kind: str, req: int):
    """(batch index, hashes, query position, extend start row or None)."""
    if kind == "ext":
        toks, p, e, start = inp.ext_meta[req]
        return req, inp.hashes[req], p, start
    toks, l = inp.dec_meta[req]
    return inp.n_ext + req, inp.hashes[inp.n_ext + req], l - 1, None


def plant_needles(run: ScenarioRun, inp: PhaseInputs, needles: list[Needle], prior: dict | None = None) -> dict:
    """Writes needle keys into the GPU inputs after ``run.store(inp)``.

    Each needle's key row is computed on the host (``needle_key`` against the
    target query's other keys, regenerated from the content generator) and
    written for its kv head at every (request, position) of the batch that
    holds the same prefix hash: the pool slot from the plan, and for an
    extend's new positions also the k_new row the extend kernel reads.
    Returns the oracle's ``key_patches`` ({prefix hash: {kv head: row}}),
    including ``prior`` patches (needles an earlier batch left in the pool).
    """
    sc = run.sc
    grp = sc.hq // sc.hkv
    patches: dict = {hh: dict(rows) for hh, rows in (prior or {}).items()}
    touched: set = set()
    kcache: dict = {}
    for nd in needles:
        bi, h, p0, _ = _req_view(inp, nd.kind, nd.req)
        qpos = p0 + (nd.row if nd.kind == "ext" else 0)
        assert 0 <= nd.pos <= qpos, (nd, qpos)
        g = nd.head // grp
        if bi not in kcache:
            kcache[bi] = cg.values(h, cg.STREAM_K, sc.hkv, sc.d)
        q = cg.values(h[qpos:qpos + 1], cg.STREAM_Q, sc.hq, sc.d, sc.q_scale_pow2)[0, nd.head]
        k = kcache[bi][:qpos + 1, g].copy()
        for hh, rows in patches.items():  # needles planted earlier in this context
            if g in rows:
                k[h[:qpos + 1] == np.uint64(hh)] = rows[g]
        others = np.delete(k, nd.pos, axis=0)
        patches.setdefault(int(h[nd.pos]), {})[g] = needle_key(q, others, sc.scale, nd.share)
        touched.add(int(h[nd.pos]))
    if not touched:
        return patches
    # every (request, position) of the batch holding a patched hash
    new = {hh: patches[hh] for hh in touched}
    keys = np.fromiter(new.keys(), dtype=np.uint64)
    kp = run.k_pool
    for bi, (h, row) in enumerate(zip(inp.hashes, inp.plan.rows)):
        hits = np.flatnonzero(np.isin(h, keys))  # the plan's row holds every position of the context
        for p in hits:
            for g, krow in new[int(h[p])].items():
                t = torch.from_numpy(krow).to(device=kp.device, dtype=torch.bfloat16)
                kp[int(row[p]), g] = t
                if bi < inp.n_ext:
                    _, pfx, _, start = inp.ext_meta[bi]
                    if p >= pfx:
                        inp.k_new[start + (p - pfx), g] = t
    torch.cuda.synchronize()
    return patches


def check_table_pool(run: ScenarioRun, inp: PhaseInputs, cpu_sample: int = 20000, seed: int = 0,
                     key_patches: dict | None = None) -> dict:
    """Table -> pool content check (bit for bit) for every attended position.

    * the device table row req_pool_idx[r] equals the plan's slot row of
      request r over its context;
    * no slot is reachable from two different prefix hashes;
    * pool[slot] holds the generator's K and V of that position's hash
      (against the GPU generator for every position, and against the CPU
      generator on a random sample); a position whose hash carries a needle
      (``key_patches``) must hold the needle's K row instead.
    """
    sc = run.sc
    table = inp.table.cpu().numpy()
    rpi = inp.rpi.cpu().numpy()
    slots_all, hashes_all = [], []
    for bi, (h, row) in enumerate(zip(inp.hashes, inp.plan.rows)):
        n = len(h)
        got = table[rpi[bi], :n]
        assert np.array_equal(got, np.asarray(row[:n], dtype=np.int32)), f"table row of request {bi}"
        slots_all.append(got.astype(np.int64))
        hashes_all.append(h)
    slots = np.concatenate(slots_all)
    hashes = np.concatenate(hashes_all)
    order = np.argsort(slots, kind="stable")
    s_sorted, h_sorted = slots[order], hashes[order]
    same_slot = s_sorted[1:] == s_sorted[:-1]
    assert not np.any(same_slot & (h_sorted[1:] != h_sorted[:-1])), "a slot is reachable from two prefix hashes"
    first = np.concatenate([[True], ~same_slot])
    u_slots, u_hashes = s_sorted[first], h_sorted[first]
    patch_keys = np.fromiter((key_patches or {}).keys(), dtype=np.uint64)
    chunk = 1 << 17
    for a in range(0, u_slots.shape[0], chunk):
        s_t = torch.from_numpy(u_slots[a:a + chunk]).to(run.k_pool.device)
        for pool, stream in ((run.k_pool, cg.STREAM_K), (run.v_pool, cg.STREAM_V)):
            exp = torch.empty((s_t.shape[0],) + tuple(pool.shape[1:]), dtype=torch.bfloat16, device=pool.device)
            gpu_gen.fill(exp, u_hashes[a:a + chunk], stream)
            if key_patches and stream == cg.STREAM_K:
                for i in np.flatnonzero(np.isin(u_hashes[a:a + chunk], patch_keys)):
                    for g, krow in key_patches[int(u_hashes[a + i])].items():
                        exp[int(i), g] = torch.from_numpy(krow).to(device=pool.device, dtype=torch.bfloat16)
            assert torch.equal(pool[s_t], exp), f"pool content differs from the generator (slots {a}..)"
    rng = np.random.default_rng(seed)
    plain = np.flatnonzero(~np.isin(u_hashes, patch_keys))
    pick = plain[rng.choice(plain.shape[0], min(cpu_sample, plain.shape[0]), replace=False)]
    s_t = torch.from_numpy(u_slots[pick]).to(run.k_pool.device)
    for pool, stream in ((run.k_pool, cg.STREAM_K), (run.v_pool, cg.STREAM_V)):
        got = pool[s_t].view(torch.int16).cpu().numpy().view(np.uint16).reshape(len(pick), -1)
        assert np.array_equal(got, cg.values_bf16_bits(u_hashes[pick], stream, sc.hkv * sc.d)), "CPU sample"
    return {"positions": int(slots.shape[0]), "distinct_slots": int(u_slots.shape[0])}


def oracle_check(run: ScenarioRun, inp: PhaseInputs, out_ext=None, out_dec=None, ext_rows=None, dec_reqs=None,
                 key_patches=None, what: str = "", workers: int | None = None) -> dict:
    """Compares kernel outputs with the oracle, requests spread over a
    process pool.  ``ext_rows``: {extend request: new-token rows} (default:
    none); ``dec_reqs``: decode requests to check (default: none).  Returns
    the worst errors per kind."""
    sc = run.sc
    tasks, keys = [], []
    for r, rows in (ext_rows or {}).items():
        toks, p, e, start = inp.ext_meta[r]
        rows = np.asarray(sorted(set(int(x) for x in rows)), dtype=np.int64)
        tasks.append(opool.extend_task(toks, p, e, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale, sc.q_scale_pow2, rows,
                                       key_patches))
        keys.append(("ext", r, start + rows))
    for r in dec_reqs or []:
        toks, l = inp.dec_meta[r]
        tasks.append(opool.decode_task(toks, l, sc.seed, sc.hq, sc.hkv, sc.d, sc.scale, sc.q_scale_pow2,
                                       key_patches))
        keys.append(("dec", r, None))
    got_e = None if out_ext is None else out_ext.float().cpu().numpy()
    got_d = None if out_dec is None else out_dec.float().cpu().numpy()
    worst = {}
    with opool.OraclePool(workers) as pool:
        for i, ref, _ in pool.imap(tasks):
            kind, r, rows = keys[i]
            got = got_e[rows] if kind == "ext" else got_d[r]
            er = assert_close(got, ref, f"{what} {kind} request {r}")
            if kind not in worst or er["max"] > worst[kind]["max"]:
                worst[kind] = dict(er, req=r)
    log(f"{what}: checked {len(tasks)} requests, worst {worst}")
    return worst
