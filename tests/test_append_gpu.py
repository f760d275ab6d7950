"""GPU parity for decode with append: this step's K/V arrive in k_new / v_new,
are written into each request's last own slot, and are attended to in the
same call.  The oracle runs on pools that hold the new token in that slot.

The slot the library writes is NaN before the call, so attending to the old
contents (instead of k_new / v_new) shows up as a non-finite result.
"""
import math
import sys

import numpy as np
import pytest
import torch

from gpu_util import assert_close, oracle_for, problem_for, to_np
from workloads import build_plan, get_config, make_batch, make_plan

pytestmark = pytest.mark.gpu

DTYPES = ["float16", "bfloat16", "float32"]


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def last_slots(plan):
    """(request, block, slot) of each request's last own token (S_r >= 1)."""
    B = plan.block_size
    out = []
    for r in range(plan.num_requests):
        S = int(plan.suffix_lens[r])
        if S > 0:
            out.append((r, int(plan.suffix_tables[r][(S - 1) // B]), (S - 1) % B))
    return out


def run_append(plan, batch, seed=7):
    """Poison the new tokens' slots, append through the library, and return
    (out, lse, pools after the call, k_new, v_new, host pools with the token)."""
    from paper_2405_19888_amd import Decoder, parrot_validate_inputs
    g = torch.Generator().manual_seed(seed)
    R, H, D = plan.num_requests, plan.heads, plan.head_dim
    td = batch.k_pool.dtype
    k_new = torch.randn((R, H, D), generator=g).to(td)
    v_new = torch.randn((R, H, D), generator=g).to(td)
    kp, vp = batch.k_pool.clone(), batch.v_pool.clone()
    kref, vref = batch.k_pool.clone(), batch.v_pool.clone()
    for r, blk, slot in last_slots(plan):
        kp[blk, :, slot] = float("nan")
        vp[blk, :, slot] = float("nan")
        kref[blk, :, slot] = k_new[r]
        vref[blk, :, slot] = v_new[r]
    dev = {k: torch.from_numpy(np.ascontiguousarray(v)).to("cuda")
           for k, v in batch.int_arrays().items()}
    dev.update(q=batch.q.to("cuda"), k_pool=kp.to("cuda"), v_pool=vp.to("cuda"),
               k_new=k_new.to("cuda"), v_new=v_new.to("cuda"))
    prob = problem_for(plan)
    scratch = torch.zeros(16, dtype=torch.int32, device="cuda")
    parrot_validate_inputs(prob, dev["prefix_tables"], dev["prefix_lens"], dev["suffix_tables"],
                           dev["suffix_lens"], dev["group_ids"], scratch)
    dec = Decoder(prob)
    dec.out.fill_(float("nan"))
    dec.lse.fill_(float("nan"))
    dec.workspace.fill_(0xFF)
    out, lse = dec(dev, append=True)
    torch.cuda.synchronize()
    return out, lse, dev, k_new, v_new, kref, vref


def append_plan(kind, dtype, D, seed=0):
    rng = np.random.default_rng(seed)
    scale = 1.0 / math.sqrt(D)
    if kind == "mixed":
        # own lengths at every slot position of the last block, S = 0, ungrouped
        gor = [0] * 6 + [1] * 5 + [-1] * 4
        sl = [1, 15, 16, 17, 0, 31, 2, 33, 48, 100, 7, 1, 16, 250, 64]
        return build_plan(heads=3, head_dim=D, block_size=16, dtype=dtype, group_of_request=gor,
                          prefix_lens=[260, 33], suffix_lens=sl, sm_scale=scale, shuffle=True,
                          rng=rng)
    if kind == "single":
        return build_plan(heads=1, head_dim=D, block_size=16, dtype=dtype, group_of_request=[-1],
                          prefix_lens=[], suffix_lens=[1], sm_scale=scale, rng=rng)
    if kind == "many_heads":
        from test_parity_gpu import many_heads_plan
        return many_heads_plan(dtype, D, rng)
    raise ValueError(kind)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("kind", ["mixed", "single", "many_heads"])
def test_append_parity(kind, dtype, D):
    say("append", kind, dtype, D)
    plan = append_plan(kind, dtype, D)
    batch = make_batch(plan, seed=3)
    out, lse, dev, k_new, v_new, kref, vref = run_append(plan, batch)
    ref = oracle_for(batch, plan, pools=(kref, vref))
    assert_close(*to_np(out, lse), *ref, dtype, f"append {kind} {dtype} D={D}")
    # the cache now holds the new token in each request's last own slot, and
    # nothing else changed
    kp, vp = dev["k_pool"].cpu(), dev["v_pool"].cpu()
    assert torch.equal(kp.nan_to_num(7.0), kref.nan_to_num(7.0))
    assert torch.equal(vp.nan_to_num(7.0), vref.nan_to_num(7.0))


def test_append_equals_write_then_decode():
    """At the LLaMA-7B one-group shape: appending gives bit for bit what the
    plain call gives on a cache that already holds the new tokens."""
    plan = make_plan(get_config("c2"))
    say(plan.num_requests, "requests, append vs write-then-decode")
    batch = make_batch(plan)
    out, lse, dev, k_new, v_new, kref, vref = run_append(plan, batch)
    a = (out.clone(), lse.clone())
    from paper_2405_19888_amd import Decoder
    dec = Decoder(problem_for(plan))
    dev2 = dict(dev, k_pool=kref.to("cuda"), v_pool=vref.to("cuda"))
    b = dec(dev2)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    reqs = [0, 7, plan.num_requests - 1]
    ref = oracle_for(batch, plan, requests=reqs, pools=(kref, vref))
    o, l = to_np(*a)
    assert_close(o[reqs], l[reqs], *ref, plan.dtype, "append c2 sampled")
