"""Batches above 1024 requests: the split-KV role streams them in slices of
1024 requests (one launch each; the prefix-group role covers every request in
the first launch, one merge follows).  2500 requests (slices 1024, 1024, 452)
mixing grouped and ungrouped requests, against the oracle, on the shared,
per-request, nested, appending and prefill entry points."""
import math
import sys

import numpy as np
import pytest
import torch

from gpu_util import assert_close, problem_for, run_gpu, run_prefill, to_np
from oracle_pool import oracle_decode, oracle_prefill
from workloads import build_plan, make_batch, make_prefill_queries

pytestmark = pytest.mark.gpu

R = 2500


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def large_plan(dtype, nested=False, seed=0):
    rng = np.random.default_rng(seed)
    # groups of 1100 (spans two slices), 700, 300 and 1 members, the rest ungrouped
    sizes = [1100, 700, 300, 1]
    gor = [g for g, n in enumerate(sizes) for _ in range(n)] + [-1] * (R - sum(sizes))
    plen = [300, 517, 64, 33]
    parents = [-1, 0, -1, 2] if nested else None
    if nested:
        plen = [304, 517, 64, 33]                 # parents fill whole blocks
    S = rng.integers(0, 90, size=R)
    S[np.asarray(gor) < 0] += 1                   # ungrouped requests need a key
    return build_plan(heads=2, head_dim=128, block_size=16, dtype=dtype, group_of_request=gor,
                      prefix_lens=plen, suffix_lens=S.tolist(), sm_scale=1 / math.sqrt(128),
                      shuffle=True, rng=rng, prefix_parents=parents)


@pytest.mark.parametrize("dtype", ["float16", "bfloat16"])
def test_decode_above_1024_requests(dtype):
    plan = large_plan(dtype)
    say("decode", R, "requests", dtype)
    batch = make_batch(plan, seed=4)
    dev = batch.to("cuda")
    res = {s: to_np(*run_gpu(plan, dev, shared=s)) for s in (True, False)}
    ref = oracle_decode(batch.q, (batch.k_pool, batch.v_pool, batch.k_pool, batch.v_pool), plan)
    for shared, (o, l) in res.items():
        assert_close(o, l, *ref, dtype, f"{R} requests shared={shared}")


def test_nested_decode_above_1024_requests():
    plan = large_plan("float16", nested=True)
    say("nested decode", R, "requests")
    batch = make_batch(plan, seed=5)
    o, l = to_np(*run_gpu(plan, batch.to("cuda")))
    ref = oracle_decode(batch.q, (batch.k_pool, batch.v_pool, batch.k_pool, batch.v_pool), plan)
    assert_close(o, l, *ref, "float16", f"nested {R} requests")


def test_append_above_1024_requests():
    """Decode with append equals writing the new tokens first, then decoding,
    bit for bit, and writes every request's new token into its slot."""
    from paper_2405_19888_amd import Decoder
    plan = large_plan("float16", seed=2)
    say("append", R, "requests")
    batch = make_batch(plan, seed=6)
    dev = batch.to("cuda")
    H, D = plan.heads, plan.head_dim
    g = torch.Generator(device="cuda").manual_seed(11)
    k_new = torch.randn((R, H, D), generator=g, device="cuda").half()
    v_new = torch.randn((R, H, D), generator=g, device="cuda").half()
    have = [r for r in range(R) if plan.suffix_lens[r] > 0]
    blk = torch.tensor([int(plan.suffix_tables[r][(int(plan.suffix_lens[r]) - 1) // 16]) for r in have],
                       device="cuda")
    slot = torch.tensor([(int(plan.suffix_lens[r]) - 1) % 16 for r in have], device="cuda")
    rows = torch.tensor(have, device="cuda")
    written = dict(dev, k_pool=dev["k_pool"].clone(), v_pool=dev["v_pool"].clone())
    written["k_pool"][blk, :, slot] = k_new[rows]
    written["v_pool"][blk, :, slot] = v_new[rows]
    ref_out, ref_lse = (t.clone() for t in run_gpu(plan, written))
    dec = Decoder(problem_for(plan))
    app = dict(dev, k_pool=dev["k_pool"].clone(), v_pool=dev["v_pool"].clone(), k_new=k_new,
               v_new=v_new)
    out, lse = dec(app, append=True)
    torch.cuda.synchronize()
    assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse)
    # bit patterns: unused slots hold NaN, which never compares equal
    for name in ("k_pool", "v_pool"):
        assert torch.equal(app[name].view(torch.int16), written[name].view(torch.int16)), name


def test_prefill_above_1024_requests(monkeypatch):
    monkeypatch.delenv("PARROT_PREFILL_SINGLE_PASS", raising=False)
    plan = large_plan("float16", seed=3)
    say("prefill", R, "requests")
    batch = make_batch(plan, seed=7)
    qr = [min(int(s), 3) for s in plan.suffix_lens]
    q, off = make_prefill_queries(plan, qr, seed=7)
    dev = batch.to("cuda")
    dev["q_rows"] = q.to("cuda")
    dev["query_offsets"] = torch.from_numpy(off).to("cuda")
    o, l = to_np(*run_prefill(plan, dev, off))
    ref = oracle_prefill(q, off, (batch.k_pool, batch.v_pool, batch.k_pool, batch.v_pool), plan)
    assert_close(o, l, *ref, "float16", f"prefill {R} requests")
