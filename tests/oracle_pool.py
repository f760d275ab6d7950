"""Run the oracle over many requests (or prefill rows) in worker processes.

The oracle is deliberately naive (each request gathers its whole context in
float64 and attends to it), so checking every request of a full-size workload
takes minutes in one process.  This helper only distributes unmodified oracle
calls, one request (or one request's rows) per task, over a pool of worker
processes that see the KV pools through shared memory.  Workers are started
with the "spawn" method (a fresh interpreter that never touches the GPU) and
run single-threaded.  No attention arithmetic here.
"""
from __future__ import annotations

import os

import numpy as np
import torch
import torch.multiprocessing as tmp

_STATE: dict = {}


def _init(state: dict) -> None:
    torch.set_num_threads(1)
    _STATE.clear()
    _STATE.update(state)


def _decode_one(r: int):
    import oracle
    s = _STATE
    out, lse = oracle.shared_prefix_decode(
        s["q"], s["pk"], s["pv"], s["sk"], s["sv"], s["ptab"], s["plen"], s["stab"], s["slen"],
        s["gid"], s["scale"], requests=[r], prefix_parents=s["parents"])
    return r, out[0], lse[0]


def _prefill_rows(rows):
    import oracle
    s = _STATE
    out, lse = oracle.shared_prefix_prefill(
        s["q"], s["qoff"], s["pk"], s["pv"], s["sk"], s["sv"], s["ptab"], s["plen"], s["stab"],
        s["slen"], s["gid"], s["scale"], rows=rows, prefix_parents=s["parents"])
    return rows, out, lse


def workers() -> int:
    """Worker processes: the CPUs this process may run on, at most 16."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def _shared(t):
    if isinstance(t, torch.Tensor):
        t = t.detach().cpu()
        if not t.is_contiguous():
            t = t.contiguous()
        t.share_memory_()
        return t
    return None if t is None else np.ascontiguousarray(t)


def _state(q, pools, plan, qoff=None) -> dict:
    pk, pv, sk, sv = (_shared(x) for x in pools)
    return dict(q=_shared(q), pk=pk, pv=pv, sk=sk, sv=sv,
                ptab=np.ascontiguousarray(plan.prefix_tables),
                plen=np.ascontiguousarray(plan.prefix_lens),
                stab=np.ascontiguousarray(plan.suffix_tables),
                slen=np.ascontiguousarray(plan.suffix_lens),
                gid=np.ascontiguousarray(plan.group_ids), scale=float(plan.sm_scale),
                parents=plan.prefix_parents if plan.nested else None,
                qoff=None if qoff is None else np.ascontiguousarray(qoff))


def oracle_decode(q, pools, plan, requests=None):
    """oracle.shared_prefix_decode for `requests` (default: all), computed in
    worker processes.  pools = (prefix_k, prefix_v, suffix_k, suffix_v), torch
    tensors on any device.  Returns (out [n, H, D], lse [n, H]) float64 in the
    order of `requests`."""
    reqs = list(range(plan.num_requests) if requests is None else requests)
    H, D = plan.heads, plan.head_dim
    out = np.zeros((len(reqs), H, D))
    lse = np.zeros((len(reqs), H))
    pos = {r: i for i, r in enumerate(reqs)}
    # longest contexts first, so the pool's tail is short
    order = sorted(reqs, key=lambda r: -int(plan.context_lens()[r]))
    ctx = tmp.get_context("spawn")
    with ctx.Pool(min(workers(), max(1, len(reqs))), initializer=_init,
                  initargs=(_state(q, pools, plan),)) as pool:
        for i, (r, o, l) in enumerate(pool.imap_unordered(_decode_one, order)):
            out[pos[r]], lse[pos[r]] = o, l
            if (i + 1) % 64 == 0:
                print(f"[oracle] {i + 1}/{len(reqs)} requests", flush=True)
    return out, lse


def oracle_prefill(q_rows, offsets, pools, plan, rows=None):
    """oracle.shared_prefix_prefill for `rows` (default: all), one task per
    request's rows (up to 64 of them), computed in worker processes.  Returns (out, lse) float64
    in the order of `rows`."""
    off = np.asarray(offsets, dtype=np.int64)
    T = int(off[-1])
    rows = list(range(T) if rows is None else rows)
    req_of = np.searchsorted(off, np.asarray(rows, dtype=np.int64), side="right") - 1
    tasks: dict[int, list] = {}
    for t, r in zip(rows, req_of):
        tasks.setdefault(int(r), []).append(int(t))
    # at most 64 rows per task (each task gathers its request's keys once)
    chunks = [rs[i:i + 64] for rs in tasks.values() for i in range(0, len(rs), 64)]
    H, D = plan.heads, plan.head_dim
    out = np.zeros((len(rows), H, D))
    lse = np.zeros((len(rows), H))
    pos = {t: i for i, t in enumerate(rows)}
    order = sorted(chunks, key=lambda x: -len(x))
    ctx = tmp.get_context("spawn")
    with ctx.Pool(min(workers(), max(1, len(order))), initializer=_init,
                  initargs=(_state(q_rows, pools, plan, qoff=off),)) as pool:
        for k, (rs, o, l) in enumerate(pool.imap_unordered(_prefill_rows, order)):
            for i, t in enumerate(rs):
                out[pos[t]], lse[pos[t]] = o[i], l[i]
            if (k + 1) % 32 == 0:
                print(f"[oracle] {k + 1}/{len(order)} row tasks", flush=True)
    return out, lse
