"""Pins for a decode-attention implementation with the oracle's signature.

Each ``pin_*`` function takes ``decode(q, prefix_k, prefix_v, suffix_k,
suffix_v, prefix_tables, prefix_lens, suffix_tables, suffix_lens, group_ids,
sm_scale, requests=None) -> (out, lse)`` and raises AssertionError when the
implementation disagrees with something the mathematics fixes independently
of it.  The oracle must pass all of them; the mutation test plants plausible
mistakes in the oracle and checks that some pin catches each one.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import torch

from workloads import build_plan, make_batch, make_plan, get_config

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def decode_args(batch, **over):
    p = batch.plan
    args = dict(q=batch.q, prefix_k=batch.k_pool, prefix_v=batch.v_pool,
                suffix_k=batch.k_pool, suffix_v=batch.v_pool,
                prefix_tables=p.prefix_tables, prefix_lens=p.prefix_lens,
                suffix_tables=p.suffix_tables, suffix_lens=p.suffix_lens,
                group_ids=p.group_ids, sm_scale=p.sm_scale)
    if p.nested:
        args["prefix_parents"] = p.prefix_parents
    args.update(over)
    return args


def tiny_paged_batch(seed=3, dtype="float32", block_size=4):
    """Two groups, an ungrouped request and a prefix-only request, paged."""
    rng = np.random.default_rng(seed)
    plan = build_plan(heads=2, head_dim=8, block_size=block_size, dtype=dtype,
                      group_of_request=[0, 0, 1, -1, 1, 0],
                      prefix_lens=[9, 5], suffix_lens=[3, 0, 7, 11, 4, 1],
                      sm_scale=1.0 / math.sqrt(8.0), paged=True, shuffle=True, rng=rng)
    return make_batch(plan, seed=seed)


def c1_batch():
    return make_batch(make_plan(get_config("tiny")))


def tiny_nested_batch(seed=4, dtype="float32", block_size=4, aligned=False):
    """Three levels of groups (0; 1 and 2 under 0; 3 under 1) with requests at
    every level, one ungrouped request, paged and shuffled.  With `aligned`,
    the prefixes that have descendants fill whole blocks."""
    rng = np.random.default_rng(seed)
    lens = [8, 4, 9, 3] if aligned else [7, 5, 9, 3]
    plan = build_plan(heads=2, head_dim=8, block_size=block_size, dtype=dtype,
                      group_of_request=[3, 3, 1, 2, 0, -1, 2, 3],
                      prefix_lens=lens, prefix_parents=[-1, 0, 0, 1],
                      suffix_lens=[2, 0, 5, 1, 4, 6, 0, 9],
                      sm_scale=1.0 / math.sqrt(8.0), paged=True, shuffle=True, rng=rng)
    return make_batch(plan, seed=seed)


def _walk_up(parents, g):
    """Brute-force chain: the groups from the outermost ancestor down to g."""
    out = []
    while g >= 0:
        out.insert(0, int(g))
        g = int(parents[g])
    return out


# ---------------------------------------------------------------- brute force
def brute_force(batch):
    """Pure-Python loops, math.exp without max shift, own index arithmetic."""
    p = batch.plan
    B = p.block_size
    q = batch.q.double().tolist()
    kp = batch.k_pool.double().tolist()
    vp = batch.v_pool.double().tolist()
    R, H, D = len(q), p.heads, p.head_dim
    outs, lses = [], []
    for r in range(R):
        keys = []   # (block, slot) of every key, prefixes first
        for g in _walk_up(p.prefix_parents, int(p.group_ids[r])):
            for t in range(int(p.prefix_lens[g])):
                keys.append((int(p.prefix_tables[g][t // B]), t % B))
        for t in range(int(p.suffix_lens[r])):
            keys.append((int(p.suffix_tables[r][t // B]), t % B))
        orow, lrow = [], []
        for h in range(H):
            es = []
            for (blk, slot) in keys:
                s = 0.0
                for d in range(D):
                    s += q[r][h][d] * kp[blk][h][slot][d]
                es.append(math.exp(p.sm_scale * s))
            z = sum(es)
            lrow.append(math.log(z))
            orow.append([sum(es[j] * vp[blk][h][slot][d] for j, (blk, slot) in enumerate(keys)) / z
                         for d in range(D)])
        outs.append(orow)
        lses.append(lrow)
    return np.array(outs), np.array(lses)


def _close(a, b, rtol, atol, what):
    a, b = np.asarray(a, dtype=np.float64), np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} != {b.shape}"
    assert np.all(np.isfinite(a)), f"{what}: non-finite values"
    err = np.abs(a - b) - (atol + rtol * np.abs(b))
    assert np.all(err <= 0), f"{what}: max excess {err.max():.3e}"


# ----------------------------------------------------------------------- pins
def pin_worked_example(decode):
    with open(os.path.join(GOLDEN, "worked_example.json")) as f:
        ex = json.load(f)
    nan = lambda x: np.array([[[[np.nan if v is None else v for v in row] for row in hb]
                               for hb in blk] for blk in x], dtype=np.float64)
    kp, vp = nan(ex["k_pool"]), nan(ex["v_pool"])
    out, lse = decode(np.array(ex["q"]), kp, vp, kp, vp, np.array(ex["prefix_tables"]),
                      np.array(ex["prefix_lens"]), np.array(ex["suffix_tables"]),
                      np.array(ex["suffix_lens"]), np.array(ex["group_ids"]), ex["sm_scale"])
    _close(out, ex["expected_out"], 0, 1e-12, "worked example out")
    _close(lse, ex["expected_lse"], 0, 1e-12, "worked example lse")


def pin_brute_force(decode):
    for batch in (c1_batch(), tiny_paged_batch(), tiny_paged_batch(seed=5, block_size=16)):
        out, lse = decode(**decode_args(batch))
        bo, bl = brute_force(batch)
        _close(out, bo, 1e-12, 1e-13, "brute force out")
        _close(lse, bl, 1e-12, 1e-13, "brute force lse")


def pin_sdpa(decode):
    batch = c1_batch()          # contiguous: identity block tables
    p = batch.plan
    out, _ = decode(**decode_args(batch))
    for r in range(p.num_requests):
        g = int(p.group_ids[r])
        P, S = int(p.prefix_lens[g]), int(p.suffix_lens[r])
        B = p.block_size
        k = batch.k_pool.double().permute(0, 2, 1, 3)   # [NB, B, H, D]
        pre = k[p.prefix_tables[g][: -(-P // B)]].reshape(-1, p.heads, p.head_dim)[:P]
        suf = k[p.suffix_tables[r][: -(-S // B)]].reshape(-1, p.heads, p.head_dim)[:S]
        v = batch.v_pool.double().permute(0, 2, 1, 3)
        vpre = v[p.prefix_tables[g][: -(-P // B)]].reshape(-1, p.heads, p.head_dim)[:P]
        vsuf = v[p.suffix_tables[r][: -(-S // B)]].reshape(-1, p.heads, p.head_dim)[:S]
        K = torch.cat([pre, suf]).permute(1, 0, 2)[None]      # [1, H, N, D]
        V = torch.cat([vpre, vsuf]).permute(1, 0, 2)[None]
        qq = batch.q.double()[r][None, :, None, :]            # [1, H, 1, D]
        ref = torch.nn.functional.scaled_dot_product_attention(qq, K, V, scale=p.sm_scale)
        _close(out[r], ref[0, :, 0, :].numpy(), 0, 1e-12, f"sdpa request {r}")


def pin_zero_query(decode):
    """q = 0: every logit is 0, so lse = ln N and out = mean of the values."""
    batch = tiny_paged_batch()
    p = batch.plan
    args = decode_args(batch, q=torch.zeros_like(batch.q))
    out, lse = decode(**args)
    N = p.context_lens()
    _close(lse, np.log(N)[:, None].repeat(p.heads, 1), 0, 1e-13, "zero-query lse")
    v = batch.v_pool.double()
    B = p.block_size
    for r in range(p.num_requests):
        acc = torch.zeros(p.heads, p.head_dim, dtype=torch.float64)
        g = int(p.group_ids[r])
        if g >= 0:
            for t in range(int(p.prefix_lens[g])):
                acc += v[int(p.prefix_tables[g][t // B]), :, t % B, :]
        for t in range(int(p.suffix_lens[r])):
            acc += v[int(p.suffix_tables[r][t // B]), :, t % B, :]
        _close(out[r], (acc / int(N[r])).numpy(), 1e-12, 1e-13, f"zero-query out {r}")


def _key_location(plan, r, j):
    g = int(plan.group_ids[r])
    B = plan.block_size
    P = int(plan.prefix_lens[g]) if g >= 0 else 0
    if j < P:
        return int(plan.prefix_tables[g][j // B]), j % B
    t = j - P
    return int(plan.suffix_tables[r][t // B]), t % B


def pin_spike(decode):
    """A key equal to c*q dominates: out = its value and lse = its logit."""
    batch = tiny_paged_batch()
    p = batch.plan
    B = p.block_size
    N = p.context_lens()
    for r in range(p.num_requests):
        g = int(p.group_ids[r])
        P = int(p.prefix_lens[g]) if g >= 0 else 0
        cand = {0, B - 1, B, P - 1, P, int(N[r]) - 1, int(N[r]) // 2}
        for j in sorted(x for x in cand if 0 <= x < int(N[r])):
            for h in range(p.heads):
                k = batch.k_pool.clone()
                blk, slot = _key_location(p, r, j)
                qv = batch.q[r, h].double()
                c = 40.0 / (p.sm_scale * float(qv @ qv))
                k[blk, h, slot, :] = (c * qv).to(k.dtype)
                out, lse = decode(**decode_args(batch, prefix_k=k, suffix_k=k),
                                  requests=[r])
                s_spike = p.sm_scale * float(batch.q[r, h].double() @ k[blk, h, slot].double())
                _close(out[0, h], batch.v_pool[blk, h, slot].double().numpy(), 0, 1e-9,
                       f"spike r={r} j={j} h={h}")
                _close(lse[0, h], s_spike, 0, 1e-9, f"spike lse r={r} j={j} h={h}")


def pin_single_and_identical_keys(decode):
    """N = 1: out = V_0, lse = s_0.  All keys equal: lse = s + ln N, out = mean V."""
    rng = np.random.default_rng(11)
    plan = build_plan(heads=2, head_dim=8, block_size=4, dtype="float32",
                      group_of_request=[0, -1, 1], prefix_lens=[1, 10],
                      suffix_lens=[0, 1, 6], sm_scale=0.5, paged=True, rng=rng)
    batch = make_batch(plan, seed=2)
    out, lse = decode(**decode_args(batch))
    for r in (0, 1):
        blk, slot = _key_location(plan, r, 0)
        s0 = 0.5 * (batch.q[r].double() * batch.k_pool[blk, :, slot].double()).sum(-1)
        _close(out[r], batch.v_pool[blk, :, slot].double().numpy(), 0, 1e-13, f"single key {r}")
        _close(lse[r], s0.numpy(), 0, 1e-13, f"single key lse {r}")
    # request 2: make all 16 of its keys identical
    k = batch.k_pool.clone()
    ref_blk, ref_slot = _key_location(plan, 2, 0)
    for j in range(16):
        blk, slot = _key_location(plan, 2, j)
        k[blk, :, slot] = batch.k_pool[ref_blk, :, ref_slot]
    out, lse = decode(**decode_args(batch, prefix_k=k, suffix_k=k), requests=[2])
    s = 0.5 * (batch.q[2].double() * k[ref_blk, :, ref_slot].double()).sum(-1)
    _close(lse[0], (s + math.log(16)).numpy(), 0, 1e-12, "identical keys lse")
    vs = torch.stack([batch.v_pool[_key_location(plan, 2, j)[0], :, _key_location(plan, 2, j)[1]]
                      for j in range(16)]).double().mean(0)
    _close(out[0], vs.numpy(), 1e-12, 1e-13, "identical keys out")


def pin_scale(decode):
    """(sigma*q, scale 1) and (q, scale sigma) give the same attention."""
    batch = tiny_paged_batch()
    sigma = batch.plan.sm_scale
    a = decode(**decode_args(batch))
    b = decode(**decode_args(batch, q=batch.q.double() * sigma, sm_scale=1.0))
    _close(a[0], b[0], 1e-11, 1e-12, "scale out")
    _close(a[1], b[1], 1e-12, 1e-12, "scale lse")


def pin_layout_invariance(decode):
    """Relabelling physical blocks changes nothing; reordering requests permutes."""
    batch = tiny_paged_batch()
    p = batch.plan
    out, lse = decode(**decode_args(batch))
    rng = np.random.default_rng(9)
    perm = rng.permutation(p.num_blocks)           # old id -> new id
    inv = np.argsort(perm)
    k2, v2 = batch.k_pool[torch.from_numpy(inv)], batch.v_pool[torch.from_numpy(inv)]
    o2, l2 = decode(**decode_args(batch, prefix_k=k2, prefix_v=v2, suffix_k=k2, suffix_v=v2,
                                  prefix_tables=perm[p.prefix_tables],
                                  suffix_tables=perm[p.suffix_tables]))
    assert np.array_equal(out, o2) and np.array_equal(lse, l2), "block relabelling changed output"
    order = rng.permutation(p.num_requests)
    o3, l3 = decode(**decode_args(batch, q=batch.q[torch.from_numpy(order)],
                                  suffix_tables=p.suffix_tables[order],
                                  suffix_lens=p.suffix_lens[order],
                                  group_ids=p.group_ids[order]))
    assert np.array_equal(out[order], o3) and np.array_equal(lse[order], l3), \
        "request reordering did not permute the output"


def pin_decomposition(decode, merge):
    """Prefix alone merged with suffix alone equals the whole context."""
    batch = tiny_paged_batch()
    p = batch.plan
    whole = decode(**decode_args(batch))
    pre = decode(**decode_args(batch, suffix_lens=np.zeros_like(p.suffix_lens)),
                 requests=[r for r in range(p.num_requests) if p.group_ids[r] >= 0])
    # suffix alone: the same requests made ungrouped
    suf = decode(**decode_args(batch, group_ids=np.full_like(p.group_ids, -1)),
                 requests=[r for r in range(p.num_requests) if p.suffix_lens[r] > 0])
    grouped = [r for r in range(p.num_requests) if p.group_ids[r] >= 0]
    withsuf = [r for r in range(p.num_requests) if p.suffix_lens[r] > 0]
    H, D = p.heads, p.head_dim
    for r in range(p.num_requests):
        parts = []
        if r in grouped:
            i = grouped.index(r)
            parts.append((pre[0][i], pre[1][i]))
        if r in withsuf:
            i = withsuf.index(r)
            parts.append((suf[0][i], suf[1][i]))
        o, l = merge(parts)
        _close(o, whole[0][r], 1e-12, 1e-12, f"decomposition out {r}")
        _close(l, whole[1][r], 1e-13, 1e-13, f"decomposition lse {r}")


def pin_nested_brute_force(decode):
    for batch in (tiny_nested_batch(), tiny_nested_batch(seed=6, block_size=16)):
        out, lse = decode(**decode_args(batch))
        bo, bl = brute_force(batch)
        _close(out, bo, 1e-12, 1e-13, "nested brute force out")
        _close(lse, bl, 1e-12, 1e-13, "nested brute force lse")


def pin_nested_zero_query(decode):
    """q = 0: lse = ln N with N the chain's prefix tokens plus the own tokens."""
    batch = tiny_nested_batch()
    p = batch.plan
    out, lse = decode(**decode_args(batch, q=torch.zeros_like(batch.q)))
    B = p.block_size
    v = batch.v_pool.double()
    for r in range(p.num_requests):
        acc = torch.zeros(p.heads, p.head_dim, dtype=torch.float64)
        n = 0
        for g in _walk_up(p.prefix_parents, int(p.group_ids[r])):
            for t in range(int(p.prefix_lens[g])):
                acc += v[int(p.prefix_tables[g][t // B]), :, t % B, :]
                n += 1
        for t in range(int(p.suffix_lens[r])):
            acc += v[int(p.suffix_tables[r][t // B]), :, t % B, :]
            n += 1
        _close(lse[r], np.full(p.heads, math.log(n)), 0, 1e-13, f"nested zero-query lse {r}")
        _close(out[r], (acc / n).numpy(), 1e-12, 1e-13, f"nested zero-query out {r}")


def pin_nested_flatten(decode):
    """Nested groups with whole-block ancestor prefixes equal flat groups whose
    tables are the chains' tables laid end to end."""
    from workloads.gen import flatten_nested
    batch = tiny_nested_batch(aligned=True)
    flat = flatten_nested(batch.plan)
    a = decode(**decode_args(batch))
    fb = type(batch)(plan=flat, q=batch.q, k_pool=batch.k_pool, v_pool=batch.v_pool)
    b = decode(**decode_args(fb))
    _close(a[0], b[0], 1e-13, 1e-14, "nested vs flattened out")
    _close(a[1], b[1], 1e-14, 1e-14, "nested vs flattened lse")


def pin_nested_spike(decode):
    """A dominant key at every level boundary of the chain."""
    batch = tiny_nested_batch()
    p = batch.plan
    B = p.block_size
    for r in range(p.num_requests):
        locs = []
        for g in _walk_up(p.prefix_parents, int(p.group_ids[r])):
            P = int(p.prefix_lens[g])
            for t in sorted({0, P - 1}):
                locs.append((int(p.prefix_tables[g][t // B]), t % B))
        S = int(p.suffix_lens[r])
        for t in sorted({0, S - 1} if S else set()):
            locs.append((int(p.suffix_tables[r][t // B]), t % B))
        for blk, slot in locs:
            h = 1
            k = batch.k_pool.clone()
            qv = batch.q[r, h].double()
            k[blk, h, slot, :] = (40.0 / (p.sm_scale * float(qv @ qv)) * qv).to(k.dtype)
            out, lse = decode(**decode_args(batch, prefix_k=k, suffix_k=k), requests=[r])
            _close(out[0, h], batch.v_pool[blk, h, slot].double().numpy(), 0, 1e-9,
                   f"nested spike r={r} block={blk} slot={slot}")


ALL_PINS = {
    "worked_example": pin_worked_example,
    "brute_force": pin_brute_force,
    "sdpa": pin_sdpa,
    "zero_query": pin_zero_query,
    "spike": pin_spike,
    "single_identical": pin_single_and_identical_keys,
    "scale": pin_scale,
    "layout_invariance": pin_layout_invariance,
    "nested_brute_force": pin_nested_brute_force,
    "nested_zero_query": pin_nested_zero_query,
    "nested_flatten": pin_nested_flatten,
    "nested_spike": pin_nested_spike,
}


# ------------------------------------------------------------------ prefill
# Pins for a prefill implementation with the signature of the oracle's
# ``shared_prefix_prefill(q, query_offsets, prefix_k, prefix_v, suffix_k,
# suffix_v, prefix_tables, prefix_lens, suffix_tables, suffix_lens, group_ids,
# sm_scale, rows=None, prefix_parents=None)``.

def prefill_args(batch, q_rows, offsets, **over):
    args = decode_args(batch, q=q_rows)
    args["query_offsets"] = offsets
    args.update(over)
    return args


def tiny_prefill_case(nested=False, seed=6):
    """(batch, q_rows, offsets): every row count from 0 to S_r (a chunk of a
    prompt whose first own tokens are already cached, a whole prompt, none)."""
    from workloads import make_prefill_queries
    batch = tiny_nested_batch(seed=seed) if nested else tiny_paged_batch(seed=seed)
    S = batch.plan.suffix_lens
    qr = [int(s) if i % 3 == 0 else int(s) // 2 if i % 3 == 1 else min(int(s), 1)
          for i, s in enumerate(S)]
    q, off = make_prefill_queries(batch.plan, qr, seed=seed)
    return batch, q, off


def _row_owner(offsets, t):
    """Brute-force: the request whose row range holds row t."""
    for r in range(len(offsets) - 1):
        if offsets[r] <= t < offsets[r + 1]:
            return r
    raise AssertionError(f"row {t} belongs to no request")


def prefill_brute_force(batch, q_rows, offsets):
    """Pure-Python loops: row t of request r is own token S_r - Q_r + (t - offsets[r])."""
    p = batch.plan
    B = p.block_size
    q = q_rows.double().tolist()
    kp = batch.k_pool.double().tolist()
    vp = batch.v_pool.double().tolist()
    outs, lses = [], []
    for t in range(len(q)):
        r = _row_owner(offsets, t)
        S = int(p.suffix_lens[r])
        Q = int(offsets[r + 1] - offsets[r])
        pos = S - Q + (t - int(offsets[r]))
        keys = []
        for g in _walk_up(p.prefix_parents, int(p.group_ids[r])):
            for j in range(int(p.prefix_lens[g])):
                keys.append((int(p.prefix_tables[g][j // B]), j % B))
        for j in range(pos + 1):
            keys.append((int(p.suffix_tables[r][j // B]), j % B))
        orow, lrow = [], []
        for h in range(p.heads):
            es = [math.exp(p.sm_scale * sum(q[t][h][d] * kp[blk][h][slot][d]
                                             for d in range(p.head_dim)))
                  for (blk, slot) in keys]
            z = sum(es)
            lrow.append(math.log(z))
            orow.append([sum(es[j] * vp[blk][h][slot][d] for j, (blk, slot) in enumerate(keys)) / z
                         for d in range(p.head_dim)])
        outs.append(orow)
        lses.append(lrow)
    return np.array(outs), np.array(lses)


def pin_prefill_brute_force(prefill):
    for nested in (False, True):
        batch, q, off = tiny_prefill_case(nested)
        out, lse = prefill(**prefill_args(batch, q, off))
        bo, bl = prefill_brute_force(batch, q, off)
        _close(out, bo, 1e-12, 1e-13, f"prefill brute force out (nested={nested})")
        _close(lse, bl, 1e-12, 1e-13, f"prefill brute force lse (nested={nested})")


def pin_prefill_sdpa(prefill):
    """torch's scaled_dot_product_attention in float64 with a boolean mask
    that lets row j see the prefix and own tokens up to its position."""
    from workloads import make_prefill_queries
    batch = c1_batch()          # contiguous: identity block tables
    p = batch.plan
    qr = [int(s) - (r % 3) if int(s) > 2 else int(s) for r, s in enumerate(p.suffix_lens)]
    q, off = make_prefill_queries(p, qr, seed=1)
    out, lse = prefill(**prefill_args(batch, q, off))
    B = p.block_size
    kk = batch.k_pool.double().permute(0, 2, 1, 3)   # [NB, B, H, D]
    vv = batch.v_pool.double().permute(0, 2, 1, 3)

    def seq(x, tbl, n):
        return x[tbl[: -(-n // B)]].reshape(-1, p.heads, p.head_dim)[:n]
    for r in range(p.num_requests):
        g = int(p.group_ids[r])
        P = int(p.prefix_lens[g]) if g >= 0 else 0
        S, Q = int(p.suffix_lens[r]), int(off[r + 1] - off[r])
        if Q == 0:
            continue
        parts_k = [seq(kk, p.prefix_tables[g], P)] if g >= 0 else []
        parts_v = [seq(vv, p.prefix_tables[g], P)] if g >= 0 else []
        K = torch.cat(parts_k + [seq(kk, p.suffix_tables[r], S)]).permute(1, 0, 2)[None]
        V = torch.cat(parts_v + [seq(vv, p.suffix_tables[r], S)]).permute(1, 0, 2)[None]
        qq = q[off[r]:off[r + 1]].double().permute(1, 0, 2)[None]     # [1, H, Q, D]
        key = torch.arange(P + S)[None, :]
        row = torch.arange(Q)[:, None]
        mask = key <= P + (S - Q) + row                                # [Q, P + S]
        ref = torch.nn.functional.scaled_dot_product_attention(qq, K, V, attn_mask=mask,
                                                               scale=p.sm_scale)
        _close(out[off[r]:off[r + 1]], ref[0].permute(1, 0, 2).numpy(), 0, 1e-12,
               f"prefill sdpa request {r}")


def pin_prefill_last_row_is_decode(prefill):
    """A request's last row sits at its last own token: it is that request's
    decode step with this row as the query (the decode pins fix that case)."""
    import oracle
    for nested in (False, True):
        batch, q, off = tiny_prefill_case(nested)
        p = batch.plan
        out, lse = prefill(**prefill_args(batch, q, off))
        last = [r for r in range(p.num_requests) if off[r + 1] > off[r]]
        qd = batch.q.clone()
        for r in last:
            qd[r] = q[int(off[r + 1]) - 1]
        do, dl = oracle.shared_prefix_decode(**decode_args(batch, q=qd), requests=last)
        rows = [int(off[r + 1]) - 1 for r in last]
        _close(out[rows], do, 1e-12, 1e-13, f"last row vs decode (nested={nested})")
        _close(lse[rows], dl, 1e-12, 1e-13, f"last row lse vs decode (nested={nested})")


def pin_prefill_causal(prefill):
    """Own tokens after a row's position change nothing (poisoned with NaN
    they stay unread); a dominant key at own position j takes over exactly the
    rows at positions >= j."""
    batch, q, off = tiny_prefill_case(False)
    p = batch.plan
    B = p.block_size
    out, lse = prefill(**prefill_args(batch, q, off))
    for r in range(p.num_requests):
        S, Q = int(p.suffix_lens[r]), int(off[r + 1] - off[r])
        if Q == 0:
            continue
        first = S - Q                                  # position of row off[r]
        k, v = batch.k_pool.clone(), batch.v_pool.clone()
        for j in range(first + 1, S):
            blk, slot = int(p.suffix_tables[r][j // B]), j % B
            k[blk, :, slot] = float("nan")
            v[blk, :, slot] = float("nan")
        o1, l1 = prefill(**prefill_args(batch, q, off, prefix_k=k, prefix_v=v, suffix_k=k,
                                        suffix_v=v), rows=[int(off[r])])
        assert np.array_equal(o1[0], out[off[r]]) and np.array_equal(l1[0], lse[off[r]]), \
            f"request {r}: a later own token changed row {off[r]}"
        j = S - 1 if Q > 1 else first                  # spike at the last own token
        blk, slot = int(p.suffix_tables[r][j // B]), j % B
        h = 0
        rows = list(range(int(off[r]), int(off[r + 1])))
        for t in rows:
            pos = first + (t - int(off[r]))
            k = batch.k_pool.clone()
            qv = q[t, h].double()
            k[blk, h, slot, :] = (40.0 / (p.sm_scale * float(qv @ qv)) * qv).to(k.dtype)
            o2, _ = prefill(**prefill_args(batch, q, off, prefix_k=k, suffix_k=k), rows=[t])
            vj = batch.v_pool[blk, h, slot].double().numpy()
            if pos >= j:
                _close(o2[0, h], vj, 0, 1e-9, f"spike at own {j} seen by row {t}")
            else:
                assert np.array_equal(o2[0, h], out[t, h]), f"row {t} saw own token {j} > {pos}"


def pin_prefill_first_row_single_key(prefill):
    """Row at own position 0 of an ungrouped request sees one key: out = V_0,
    lse = s_0."""
    from workloads import make_prefill_queries
    batch = tiny_paged_batch()
    p = batch.plan
    qr = [int(s) if int(p.group_ids[r]) < 0 else 0 for r, s in enumerate(p.suffix_lens)]
    q, off = make_prefill_queries(p, qr, seed=3)
    out, lse = prefill(**prefill_args(batch, q, off))
    B = p.block_size
    for r in range(p.num_requests):
        if qr[r] == 0:
            continue
        t = int(off[r])
        blk, slot = int(p.suffix_tables[r][0]), 0
        s0 = p.sm_scale * (q[t].double() * batch.k_pool[blk, :, slot].double()).sum(-1)
        _close(out[t], batch.v_pool[blk, :, slot].double().numpy(), 0, 1e-13, f"first row {t}")
        _close(lse[t], s0.numpy(), 0, 1e-13, f"first row lse {t}")


PREFILL_PINS = {
    "prefill_brute_force": pin_prefill_brute_force,
    "prefill_sdpa": pin_prefill_sdpa,
    "prefill_last_row_is_decode": pin_prefill_last_row_is_decode,
    "prefill_causal": pin_prefill_causal,
    "prefill_first_row_single_key": pin_prefill_first_row_single_key,
}
