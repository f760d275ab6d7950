"""Seeded random plans against the float64 oracle: decode (flat groups on both
paths, nested chains on the nested entry point), decode with append, and
prefill (both plans).

Each seed draws the head count, head size, cache type, softmax scale (unit
or half, either sign), group structure (empty groups, groups above one
64-query tile, ungrouped requests) and lengths with a bias towards the edges
that the kernels cut at (block, stage and chunk boundaries, one token, empty
own ranges).  The cases are small, so the whole output is compared with the
oracle.
"""
import math
import sys

import numpy as np
import pytest

from gpu_util import (assert_close, oracle_for, oracle_prefill_for, run_gpu, run_prefill, to_np)
from workloads import build_plan, make_batch, make_prefill_queries

pytestmark = pytest.mark.gpu

DTYPES = ["float16", "bfloat16", "float32"]
EDGES = [1, 15, 16, 17, 31, 32, 33, 255, 256, 257, 511, 512, 513]


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def draw_len(rng, hi, lo=0):
    """A length in [lo, hi]: an edge value half of the time, else uniform."""
    if rng.random() < 0.5:
        e = [x for x in EDGES + [lo] if lo <= x <= hi]
        return int(rng.choice(e))
    return int(rng.integers(lo, hi + 1))


def random_plan(seed, nested):
    rng = np.random.default_rng(10_000 + seed)
    dtype = DTYPES[seed % 3]
    D = (64, 128)[(seed // 3) % 2]
    H = int(rng.integers(1, 9))
    # unit-scale logits or smaller, either sign: the tolerance bars are derived
    # for unit-scale logits (a peaked softmax over bf16-rounded weights can
    # exceed them); large logits have tests of their own (the logit ramps)
    scale = float(rng.choice([1.0, -1.0, 0.5])) / math.sqrt(D)
    NG = int(rng.integers(1 if nested else 0, 5))
    R = int(rng.integers(1, 14))
    gor = [int(rng.integers(-1, NG)) if NG else -1 for _ in range(R)]
    if NG and max(gor) < 0:
        gor[0] = 0                                      # at least one grouped request
    if rng.random() < 0.3 and NG:
        gor += [0] * int(rng.integers(60, 80))         # a group above one 64-query tile
    R = len(gor)
    plen = [draw_len(rng, 1200, 1) for _ in range(NG)]
    sl = [draw_len(rng, 700) for _ in range(R)]
    # every request needs at least one key
    sl = [max(s, 1) if g < 0 else s for s, g in zip(sl, gor)]
    parents = None
    if nested:
        # a forest: each group's parent is an earlier group or none, depth <= 4
        parents, depth = [], []
        for g in range(NG):
            cands = [p for p in range(g) if depth[p] < 3]
            p = int(rng.choice(cands)) if cands and rng.random() < 0.7 else -1
            parents.append(p)
            depth.append(0 if p < 0 else depth[p] + 1)
    plan = build_plan(heads=H, head_dim=D, block_size=16, dtype=dtype, group_of_request=gor,
                      prefix_lens=plen, suffix_lens=sl, sm_scale=scale, shuffle=True, rng=rng,
                      prefix_parents=parents)
    return plan, rng


@pytest.mark.parametrize("seed", range(18))
def test_random_decode(seed):
    plan, _ = random_plan(seed, nested=False)
    say("random decode", seed, plan.dtype, "D", plan.head_dim, "H", plan.heads, "R",
        plan.num_requests, "groups", plan.num_groups, "scale", round(plan.sm_scale, 4))
    batch = make_batch(plan, seed=seed)
    dev = batch.to("cuda")
    ref = oracle_for(batch, plan)
    for shared in (True, False):
        out, lse = run_gpu(plan, dev, shared=shared)
        assert_close(*to_np(out, lse), *ref, plan.dtype, f"seed {seed} shared={shared}")


@pytest.mark.parametrize("seed", range(12))
def test_random_nested_decode(seed):
    plan, _ = random_plan(seed, nested=True)
    say("random nested decode", seed, plan.dtype, "D", plan.head_dim, "H", plan.heads, "R",
        plan.num_requests, "parents", list(plan.prefix_parents))
    batch = make_batch(plan, seed=seed)
    out, lse = run_gpu(plan, batch.to("cuda"))
    assert_close(*to_np(out, lse), *oracle_for(batch, plan), plan.dtype, f"nested seed {seed}")


@pytest.mark.parametrize("plan_path", ["split", "single"])
@pytest.mark.parametrize("seed", range(12))
def test_random_prefill(seed, plan_path, monkeypatch):
    plan, rng = random_plan(seed, nested=False)
    if plan_path == "single" and plan.dtype == "float32":
        plan_path = "split"                  # the single pass serves 16-bit caches
    monkeypatch.setenv("PARROT_PREFILL_SINGLE_PASS", "1" if plan_path == "single" else "0")
    # rows per request: the whole prompt, none, one, or a random tail
    qr = []
    for s in plan.suffix_lens:
        s = int(s)
        c = rng.random()
        qr.append(s if c < 0.3 else 0 if c < 0.45 else min(1, s) if c < 0.6 else int(rng.integers(0, s + 1)))
    say("random prefill", seed, plan_path, plan.dtype, "D", plan.head_dim, "H", plan.heads,
        "rows", sum(qr))
    batch = make_batch(plan, seed=seed)
    q, off = make_prefill_queries(plan, qr, seed=seed)
    dev = batch.to("cuda")
    import torch
    dev["q_rows"] = q.to("cuda")
    dev["query_offsets"] = torch.from_numpy(np.ascontiguousarray(off)).to("cuda")
    out, lse = run_prefill(plan, dev, off)
    ref = oracle_prefill_for(batch, plan, q, off)
    assert_close(*to_np(out, lse), *ref, plan.dtype, f"prefill seed {seed} {plan_path}")


@pytest.mark.parametrize("seed", range(10))
def test_random_append(seed):
    """Decode with append on random flat plans: the output against the oracle
    on pools that hold each request's new token, and the cache afterwards."""
    import torch
    from test_append_gpu import run_append
    plan, _ = random_plan(seed, nested=False)
    say("random append", seed, plan.dtype, "D", plan.head_dim, "H", plan.heads, "R",
        plan.num_requests)
    batch = make_batch(plan, seed=seed)
    out, lse, dev, k_new, v_new, kref, vref = run_append(plan, batch, seed=seed)
    ref = oracle_for(batch, plan, pools=(kref, vref))
    assert_close(*to_np(out, lse), *ref, plan.dtype, f"append seed {seed}")
    assert torch.equal(dev["k_pool"].cpu().nan_to_num(7.0), kref.nan_to_num(7.0))
    assert torch.equal(dev["v_pool"].cpu().nan_to_num(7.0), vref.nan_to_num(7.0))
