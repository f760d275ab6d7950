"""GPU parity: the HIP library (through its C ABI) against the float64 oracle.

Every case prints its name before touching the GPU, validates the device-side
inputs with parrot_validate_inputs, NaN-poisons the outputs and the workspace,
and compares element by element.
"""
import math
import sys

import numpy as np
import pytest
import torch

from gpu_util import assert_close, oracle_for, problem_for, run_gpu, to_np
from workloads import build_plan, get_config, make_batch, make_plan

pytestmark = pytest.mark.gpu

DTYPES = ["float16", "bfloat16", "float32"]


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


# ------------------------------------------------------------------ workloads
@pytest.mark.parametrize("shared", [True, False], ids=["shared", "per_request"])
@pytest.mark.parametrize("name", ["c1", "c2"])
def test_config_full_parity(name, shared):
    cfg = get_config(name)
    say(name, cfg.name, "shared" if shared else "per_request")
    plan = make_plan(cfg)
    batch = make_batch(plan)
    out, lse = run_gpu(plan, batch.to("cuda"), shared=shared)
    ref = oracle_for(batch, plan)
    assert_close(*to_np(out, lse), *ref, plan.dtype, f"{cfg.name} shared={shared}")


# The shared-system-prompt, map-reduce and 32-layer mixed workloads are
# compared request by request with the oracle in test_fullsize_gpu.py.


# ----------------------------------------------------------------- edge cases
def edge_plan(kind, dtype, D, seed=0):
    rng = np.random.default_rng(seed)
    scale = 1.0 / math.sqrt(D)
    if kind == "boundaries":
        # groups of 3, 17 and 1 members; prefix lengths at chunk/block edges;
        # suffix lengths at block and chunk edges, including 0; two ungrouped
        gor = [0] * 3 + [1] * 17 + [2] + [-1, -1]
        plen = [1, 257, 16]
        sl = [0, 1, 15, 16, 17, 127, 128, 129, 255, 256, 257, 0, 3, 31, 33, 64, 100, 2, 5, 9,
              129, 1, 300]
        return build_plan(heads=3, head_dim=D, block_size=16, dtype=dtype, group_of_request=gor,
                          prefix_lens=plen, suffix_lens=sl, sm_scale=scale, shuffle=True, rng=rng)
    if kind == "big_group":
        n = 130
        return build_plan(heads=2, head_dim=D, block_size=16, dtype=dtype,
                          group_of_request=[0] * n, prefix_lens=[40],
                          suffix_lens=rng.integers(0, 40, size=n).tolist(), sm_scale=scale,
                          shuffle=True, rng=rng)
    if kind == "ungrouped":
        return build_plan(heads=4, head_dim=D, block_size=16, dtype=dtype,
                          group_of_request=[-1] * 5, prefix_lens=[],
                          suffix_lens=[1, 16, 200, 513, 7], sm_scale=scale, rng=rng)
    if kind == "single_key":
        return build_plan(heads=1, head_dim=D, block_size=16, dtype=dtype, group_of_request=[0],
                          prefix_lens=[1], suffix_lens=[0], sm_scale=scale, rng=rng)
    if kind == "chunk_multiples":
        return build_plan(heads=2, head_dim=D, block_size=16, dtype=dtype,
                          group_of_request=[0, 0, 1, 1, 1], prefix_lens=[256, 512],
                          suffix_lens=[128, 256, 0, 384, 16], sm_scale=scale, shuffle=True, rng=rng)
    if kind == "long_prefix_4g":
        # enough prefix work (max prefix x groups x heads = 5000 x 4 x 8) that
        # the prefix chunk grows past 256 tokens (1024 on a 256-CU device)
        gor = [0, 0, 1, 2, 2, 3, -1]
        return build_plan(heads=8, head_dim=D, block_size=16, dtype=dtype, group_of_request=gor,
                          prefix_lens=[5000, 511, 513, 1537],
                          suffix_lens=rng.integers(0, 90, size=len(gor)).tolist(), sm_scale=scale,
                          shuffle=True, rng=rng)
    if kind == "long_prefix_8g":
        # 4200 x 8 x 8: a 512-token prefix chunk on a 256-CU device
        gor = [g for g in range(8) for _ in range(2)]
        return build_plan(heads=8, head_dim=D, block_size=16, dtype=dtype, group_of_request=gor,
                          prefix_lens=[4200, 1025, 1023, 3000, 17, 2049, 4096, 700],
                          suffix_lens=rng.integers(0, 100, size=len(gor)).tolist(), sm_scale=scale,
                          shuffle=True, rng=rng)
    if kind == "many_heads":
        return many_heads_plan(dtype, D, rng)
    raise ValueError(kind)


def many_heads_plan(dtype, D, rng):
    """128 heads (16 split-KV waves per head on a 256-CU device): long runs of
    the flat column list that cross many requests; ragged lengths, two groups
    and ungrouped requests."""
    gor = [0] * 12 + [1] * 12 + [-1] * 12
    sl = rng.integers(150, 400, size=len(gor)).tolist()
    sl[5], sl[30] = 0, 1
    return build_plan(heads=128, head_dim=D, block_size=16, dtype=dtype, group_of_request=gor,
                      prefix_lens=[300, 1000], suffix_lens=sl, sm_scale=1.0 / math.sqrt(D),
                      shuffle=True, rng=rng)


EDGE_KINDS = ["boundaries", "big_group", "ungrouped", "single_key", "chunk_multiples",
              "long_prefix_4g", "long_prefix_8g", "many_heads"]


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("kind", EDGE_KINDS)
def test_edge_cases(kind, dtype, D):
    say("edge", kind, dtype, D)
    plan = edge_plan(kind, dtype, D)
    batch = make_batch(plan, seed=1)
    dev = batch.to("cuda")
    ref = oracle_for(batch, plan)
    for shared in (True, False):
        out, lse = run_gpu(plan, dev, shared=shared)
        assert_close(*to_np(out, lse), *ref, dtype, f"{kind} {dtype} D={D} shared={shared}")


def test_empty_batch_is_noop():
    say("empty batch")
    plan = edge_plan("ungrouped", "float16", 128)
    prob = problem_for(plan)
    prob.num_requests = 0
    from paper_2405_19888_amd import parrot_shared_prefix_decode
    z = torch.zeros(16, dtype=torch.float16, device="cuda")
    zi = torch.zeros(4, dtype=torch.int32, device="cuda")
    parrot_shared_prefix_decode(prob, z, z, z, z, z, zi, zi, zi, zi, zi, z, None, None)
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype", ["float16", "bfloat16"])
def test_separate_prefix_and_suffix_pools(dtype):
    """Prefix blocks are read from the prefix pools only, suffix blocks from the
    suffix pools only: each pool has the other's blocks set to NaN."""
    say("separate pools", dtype)
    plan = edge_plan("boundaries", dtype, 128)
    batch = make_batch(plan, seed=2)
    dev = batch.to("cuda")
    pre_blocks = set(int(x) for g in range(plan.num_groups)
                     for x in plan.prefix_tables[g][: -(-int(plan.prefix_lens[g]) // 16)])
    pre_idx = torch.tensor(sorted(pre_blocks), device="cuda")
    suf_mask = torch.ones(plan.num_blocks, dtype=torch.bool, device="cuda")
    suf_mask[pre_idx] = False
    pk, pv = dev["k_pool"].clone(), dev["v_pool"].clone()
    sk, sv = dev["k_pool"].clone(), dev["v_pool"].clone()
    pk[suf_mask] = float("nan"); pv[suf_mask] = float("nan")
    sk[pre_idx] = float("nan"); sv[pre_idx] = float("nan")
    dev2 = dict(dev, prefix_k=pk, prefix_v=pv, suffix_k=sk, suffix_v=sv)
    ref = oracle_for(batch, plan)
    for shared in (True, False):
        out, lse = run_gpu(plan, dev2, shared=shared)
        assert_close(*to_np(out, lse), *ref, dtype, f"separate pools shared={shared}")


# --------------------------------------------------------------------- probes
def probe_plan(dtype):
    rng = np.random.default_rng(7)
    return build_plan(heads=2, head_dim=128, block_size=16, dtype=dtype,
                      group_of_request=[0, 0, 0, -1], prefix_lens=[530],
                      suffix_lens=[300, 0, 17, 260], sm_scale=1 / math.sqrt(128), shuffle=False,
                      rng=rng)


@pytest.mark.parametrize("dtype", ["float16", "bfloat16"])
def test_zero_query_probe(dtype):
    """q = 0: lse = ln N exactly and out = mean of the N values (pins lengths)."""
    say("zero-query probe", dtype)
    plan = probe_plan(dtype)
    batch = make_batch(plan, seed=3)
    batch.q.zero_()
    dev = batch.to("cuda")
    ref_out, ref_lse = oracle_for(batch, plan)
    N = plan.context_lens()
    assert np.allclose(ref_lse, np.log(N)[:, None], rtol=1e-12, atol=0)
    for shared in (True, False):
        out, lse = run_gpu(plan, dev, shared=shared)
        o, l = to_np(out, lse)
        assert np.max(np.abs(l - ref_lse) / ref_lse) < 1e-6, f"shared={shared}"
        assert np.max(np.abs(o - ref_out)) < (4e-3 if dtype == "bfloat16" else 5e-4)


@pytest.mark.parametrize("dtype", ["float16", "bfloat16"])
def test_spike_probe(dtype):
    """A key c*q with logit 40 dominates: out = its value, lse = its logit.
    Positions cover block, prefix-chunk, suffix-chunk and sequence edges."""
    say("spike probe", dtype)
    plan = probe_plan(dtype)
    base = make_batch(plan, seed=4)
    B = 16
    for r in (0, 3):
        g = int(plan.group_ids[r])
        P = int(plan.prefix_lens[g]) if g >= 0 else 0
        N = int(plan.context_lens()[r])
        for j in sorted({0, 15, 16, 255, 256, P - 1, P, P + 127, P + 128, N - 1}):
            if not 0 <= j < N:
                continue
            k = base.k_pool.clone()
            if j < P:
                blk, slot = int(plan.prefix_tables[g][j // B]), j % B
            else:
                t = j - P
                blk, slot = int(plan.suffix_tables[r][t // B]), t % B
            for h in range(plan.heads):
                qv = base.q[r, h].double()
                c = 40.0 / (plan.sm_scale * float(qv @ qv))
                k[blk, h, slot] = (c * qv).to(k.dtype)
            batch = type(base)(plan=plan, q=base.q, k_pool=k, v_pool=base.v_pool)
            dev = batch.to("cuda")
            for shared in (True, False):
                out, lse = run_gpu(plan, dev, shared=shared)
                o, l = to_np(out, lse)
                v = base.v_pool[blk, :, slot].double().numpy()
                s = plan.sm_scale * (base.q[r].double() * k[blk, :, slot].double()).sum(-1).numpy()
                assert np.max(np.abs(o[r] - v)) <= 1e-3 * max(1.0, np.abs(v).max()), \
                    f"spike r={r} j={j} shared={shared}"
                assert np.max(np.abs(l[r] - s) / np.abs(s)) < 1e-5, f"spike lse r={r} j={j}"


# ------------------------------------------------------ scale and logit range
def scale_plan(dtype, sm_scale):
    """Groups of 70 (two 64-query tiles), 5 and 1 members over prefixes long
    enough for many stages, plus two ungrouped requests."""
    rng = np.random.default_rng(11)
    gor = [0] * 70 + [1] * 5 + [2] + [-1, -1]
    return build_plan(heads=2, head_dim=128, block_size=16, dtype=dtype, group_of_request=gor,
                      prefix_lens=[1500, 700, 33],
                      suffix_lens=rng.integers(0, 120, size=len(gor)).tolist(), sm_scale=sm_scale,
                      shuffle=True, rng=rng)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("kind", ["negative_scale", "zero_scale", "ramp"])
def test_scale_and_logit_range(kind, dtype):
    """sm_scale < 0 and sm_scale = 0, and logits that climb along a long prefix
    (the softmax reference moves again and again within a chunk), against the
    oracle on both paths."""
    say("scale / logit range", kind, dtype)
    D = 128
    scale = {"negative_scale": -1 / math.sqrt(D), "zero_scale": 0.0, "ramp": 1 / math.sqrt(D)}[kind]
    plan = scale_plan(dtype, scale)
    batch = make_batch(plan, seed=5)
    if kind == "ramp":
        # group 0's members share a query direction u (plus noise); its prefix key
        # j is ramp_j / (scale |u|^2) u plus noise, so every member's logit of key j
        # is about ramp_j, climbing from 0 to 200 over the prefix: about 17 per
        # 128-token chunk, several moves of a lazily kept reference per chunk
        g = 0
        P = int(plan.prefix_lens[g])
        td = batch.q.dtype
        q = batch.q.float()
        k = batch.k_pool.float()
        u = torch.randn((plan.heads, D), generator=torch.Generator().manual_seed(9))
        for r in np.flatnonzero(plan.group_ids == g):
            q[r] = u + 0.05 * q[r]
        for j in range(P):
            blk, slot = int(plan.prefix_tables[g][j // plan.block_size]), j % plan.block_size
            for h in range(plan.heads):
                c = 200.0 * j / P / (scale * float(u[h] @ u[h]))
                k[blk, h, slot] = c * u[h] + 0.05 * k[blk, h, slot]
        batch = type(batch)(plan=plan, q=q.to(td), k_pool=k.to(td), v_pool=batch.v_pool)
    # fp32 caches: a logit near 200 carries a rounding error of about
    # sqrt(D) 2^-24 200 = 1.4e-4 from its fp32 dot product, and so does each
    # weight relatively; with |v| up to about 4 that bounds the output error by
    # 6e-4 (relative L2 by 2e-4), above the 1e-5 kept for unit-scale logits
    loose = kind == "ramp" and dtype == "float32"
    ref = oracle_for(batch, plan)
    dev = batch.to("cuda")
    for shared in (True, False):
        out, lse = run_gpu(plan, dev, shared=shared)
        assert_close(*to_np(out, lse), *ref, dtype, f"{kind} {dtype} shared={shared}",
                     out_tol=6e-4 if loose else None, rel_l2=2e-4 if loose else None)


# ------------------------------------------------------------ other properties
def test_bitwise_reproducible():
    say("reproducibility")
    plan = make_plan(get_config("c2"))
    dev = make_batch(plan).to("cuda")
    a = [t.clone() for t in run_gpu(plan, dev)]
    b = run_gpu(plan, dev)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_validate_inputs_reports_bad_entries():
    say("validate")
    from paper_2405_19888_amd import ParrotError, parrot_validate_inputs
    plan = edge_plan("boundaries", "float16", 128)
    dev = make_batch(plan).to("cuda")
    prob = problem_for(plan)
    scratch = torch.zeros(16, dtype=torch.int32, device="cuda")
    parrot_validate_inputs(prob, dev["prefix_tables"], dev["prefix_lens"], dev["suffix_tables"],
                           dev["suffix_lens"], dev["group_ids"], scratch)
    bad = dev["suffix_tables"].clone()
    r = int(np.argmax(plan.suffix_lens))
    bad[r, 0] = plan.num_blocks + 5
    with pytest.raises(ParrotError, match="suffix block id"):
        parrot_validate_inputs(prob, dev["prefix_tables"], dev["prefix_lens"], bad,
                               dev["suffix_lens"], dev["group_ids"], scratch)
    badg = dev["group_ids"].clone()
    badg[1] = plan.num_groups
    with pytest.raises(ParrotError, match="group id"):
        parrot_validate_inputs(prob, dev["prefix_tables"], dev["prefix_lens"], dev["suffix_tables"],
                               dev["suffix_lens"], badg, scratch)


def test_validate_inputs_reports_group_above_max_group_size():
    """A group read by 65 requests under max_group_size = 64: the prefix role
    sizes its query tiles from the bound, so the validator must refuse it."""
    say("validate max_group_size")
    from paper_2405_19888_amd import ParrotError, parrot_validate_inputs
    rng = np.random.default_rng(11)
    plan = build_plan(heads=2, head_dim=128, block_size=16, dtype="float16",
                      group_of_request=[0] * 65 + [-1], prefix_lens=[40],
                      suffix_lens=rng.integers(1, 30, size=66).tolist(),
                      sm_scale=1 / math.sqrt(128), shuffle=True, rng=rng)
    dev = make_batch(plan).to("cuda")
    prob = problem_for(plan)
    scratch = torch.zeros(16, dtype=torch.int32, device="cuda")
    args = (dev["prefix_tables"], dev["prefix_lens"], dev["suffix_tables"], dev["suffix_lens"],
            dev["group_ids"], scratch)
    assert prob.max_group_size == 65
    parrot_validate_inputs(prob, *args)
    prob.max_group_size = 64
    with pytest.raises(ParrotError, match="max_group_size") as e:
        parrot_validate_inputs(prob, *args)
    assert e.value.status == 1


def test_trace_events_time_each_kernel():
    say("trace events")
    from paper_2405_19888_amd import Decoder, ParrotTrace
    plan = make_plan(get_config("c2"))
    dev = make_batch(plan).to("cuda")
    dec = Decoder(problem_for(plan))
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in evs:
        e.record()
    torch.cuda.synchronize()
    tr = ParrotTrace(*[e.cuda_event for e in evs])
    dec(dev, shared=True, trace=tr)
    torch.cuda.synchronize()
    times = [evs[2 * i].elapsed_time(evs[2 * i + 1]) for i in range(2)]
    assert all(t > 0 for t in times), times
    assert evs[1].elapsed_time(evs[2]) >= 0        # the merge runs after the partials


@pytest.mark.parametrize("per_request", [False, True])
def test_one_call_torch_api(per_request):
    """shared_prefix_decode on plain torch tensors sizes the problem itself and
    matches the oracle (flat groups, ungrouped requests, separate pools)."""
    from paper_2405_19888_amd import shared_prefix_decode
    say("one-call torch API, per_request =", per_request)
    plan = edge_plan("boundaries", "float16", 128)
    batch = make_batch(plan, seed=2)
    dev = batch.to("cuda")
    out, lse = shared_prefix_decode(
        dev["q"], dev["k_pool"], dev["v_pool"], dev["k_pool"], dev["v_pool"], dev["prefix_tables"],
        dev["prefix_lens"], dev["suffix_tables"], dev["suffix_lens"], dev["group_ids"],
        sm_scale=plan.sm_scale, per_request=per_request)
    torch.cuda.synchronize()
    ref = oracle_for(batch, plan)
    assert_close(*to_np(out, lse), *ref, "float16", f"one-call per_request={per_request}")
