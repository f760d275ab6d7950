"""GPU parity for nested prefix groups: the HIP library (through its C ABI)
against the float64 oracle, which reads each request's chain of prefixes
outermost first, then its own tokens.

Every case prints its name before touching the GPU and validates the device
inputs (parents included) before the call; outputs and workspace are
NaN-poisoned first.
"""
import math
import sys

import numpy as np
import pytest
import torch

from gpu_util import assert_close, oracle_for, problem_for, run_gpu, to_np
from workloads import build_plan, get_config, make_batch, make_device_layer, make_plan
from workloads.gen import flatten_nested

pytestmark = pytest.mark.gpu

DTYPES = ["float16", "bfloat16", "float32"]


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def nested_plan(kind, dtype, D, seed=0):
    rng = np.random.default_rng(seed)
    scale = 1.0 / math.sqrt(D)
    if kind == "four_levels":
        # 0 <- 1 <- 3 <- 4 and 0 <- 2; requests at every level and ungrouped
        gor = [4] * 5 + [3] * 3 + [1] * 4 + [2] * 6 + [0] * 2 + [-1] * 2
        return build_plan(heads=3, head_dim=D, block_size=16, dtype=dtype, group_of_request=gor,
                          prefix_lens=[700, 130, 257, 33, 16], prefix_parents=[-1, 0, 0, 1, 3],
                          suffix_lens=rng.integers(0, 200, size=len(gor)).tolist(),
                          sm_scale=scale, shuffle=True, rng=rng)
    if kind == "wide_root":
        # 96 requests read the root's prefix: two 64-query tiles
        gor = [g for g in range(1, 7) for _ in range(16)]
        return build_plan(heads=2, head_dim=D, block_size=16, dtype=dtype, group_of_request=gor,
                          prefix_lens=[300, 50, 64, 17, 1, 99, 80],
                          prefix_parents=[-1, 0, 0, 0, 0, 0, 0],
                          suffix_lens=rng.integers(0, 70, size=len(gor)).tolist(),
                          sm_scale=scale, shuffle=True, rng=rng)
    if kind == "forest":
        # two trees; members at both roots; group 6 has no readers
        gor = [0, 0, 2, 2, 2, 3, 1, 4, 4, 5]
        return build_plan(heads=4, head_dim=D, block_size=16, dtype=dtype, group_of_request=gor,
                          prefix_lens=[512, 16, 200, 31, 600, 7, 40],
                          prefix_parents=[-1, -1, 0, 2, 1, 4, 0],
                          suffix_lens=[0, 5, 40, 0, 300, 1, 17, 64, 3, 128],
                          sm_scale=scale, shuffle=True, rng=rng)
    if kind == "long_root":
        # a root long enough for several prefix chunks under children
        gor = [1] * 5 + [2] * 5 + [3] * 5
        return build_plan(heads=8, head_dim=D, block_size=16, dtype=dtype, group_of_request=gor,
                          prefix_lens=[4100, 256, 1000, 16], prefix_parents=[-1, 0, 0, 2],
                          suffix_lens=rng.integers(1, 120, size=len(gor)).tolist(),
                          sm_scale=scale, shuffle=True, rng=rng)
    raise ValueError(kind)


KINDS = ["four_levels", "wide_root", "forest", "long_root"]


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("kind", KINDS)
def test_nested_parity(kind, dtype, D):
    say("nested", kind, dtype, D)
    plan = nested_plan(kind, dtype, D)
    batch = make_batch(plan, seed=2)
    out, lse = run_gpu(plan, batch.to("cuda"))
    assert_close(*to_np(out, lse), *oracle_for(batch, plan), dtype, f"nested {kind} {dtype} D={D}")


def test_nested_entry_with_flat_groups_matches_flat_entry():
    say("nested entry, all parents -1")
    rng = np.random.default_rng(5)
    plan = build_plan(heads=4, head_dim=128, block_size=16, dtype="float16",
                      group_of_request=[0, 0, 1, 1, 1, -1], prefix_lens=[300, 45],
                      suffix_lens=[3, 90, 0, 17, 200, 33], sm_scale=1 / math.sqrt(128),
                      shuffle=True, rng=rng)
    dev = make_batch(plan).to("cuda")
    a = [t.clone() for t in run_gpu(plan, dev, nested=False)]
    b = run_gpu(plan, dev, nested=True)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_nested_system_prompt_workload():
    """The two-level workload at full size: every request against the oracle;
    as an extra, every request against the flat entry points run on the same
    blocks with each sub-group's chain laid end to end."""
    from oracle_pool import oracle_decode
    cfg = get_config("nested")
    plan = make_plan(cfg)
    say(cfg.name, "requests", plan.num_requests)
    batch = make_batch(plan)
    dev = batch.to("cuda")
    out, lse = run_gpu(plan, dev)
    o, l = to_np(out, lse)
    ref = oracle_decode(batch.q, (batch.k_pool, batch.v_pool, batch.k_pool, batch.v_pool), plan)
    assert_close(o, l, *ref, plan.dtype, "nested workload, every request")
    flat = flatten_nested(plan)
    fdev = dict(dev)
    for k, v in (("prefix_tables", flat.prefix_tables), ("prefix_lens", flat.prefix_lens),
                 ("group_ids", flat.group_ids), ("prefix_parents", flat.prefix_parents)):
        fdev[k] = torch.from_numpy(np.ascontiguousarray(v)).to("cuda")
    for shared in (True, False):
        say(cfg.name, "flattened", "shared" if shared else "per_request")
        fo, fl = to_np(*run_gpu(flat, fdev, shared=shared))
        assert np.all(np.isfinite(o)) and np.all(np.isfinite(l))
        assert np.max(np.abs(o - fo)) <= 2e-3
        assert np.max(np.abs(l - fl) / np.maximum(1, np.abs(fl))) <= 1e-4


def test_nested_validation_rejects_bad_parents():
    say("nested validation")
    from paper_2405_19888_amd import ParrotError, parrot_validate_nested_inputs
    plan = nested_plan("four_levels", "float16", 128)
    dev = make_batch(plan).to("cuda")
    prob = problem_for(plan)
    scratch = torch.zeros(16, dtype=torch.int32, device="cuda")
    args = lambda par: (prob, dev["prefix_tables"], dev["prefix_lens"], par, dev["suffix_tables"],
                        dev["suffix_lens"], dev["group_ids"], scratch)
    parrot_validate_nested_inputs(*args(dev["prefix_parents"]))
    bad = dev["prefix_parents"].clone()
    bad[1] = 3                                   # a parent that is not a lower group
    with pytest.raises(ParrotError, match="prefix parent|deeper than"):
        parrot_validate_nested_inputs(*args(bad))
    prob.max_prefix_depth = 3                    # the chain 0 <- 1 <- 3 <- 4 has 4 groups
    with pytest.raises(ParrotError, match="deeper"):
        parrot_validate_nested_inputs(*args(dev["prefix_parents"]))


def plan_from_store(batch, store, heads, head_dim, dtype):
    """A LayoutPlan over the store's blocks (block num_blocks is the NaN pad)."""
    from workloads.gen import LayoutPlan
    B, NB = store.block_size, store.num_blocks + 1
    fill = np.zeros(NB, dtype=np.int32)
    for lens, tabs in ((batch.prefix_lens, batch.prefix_tables),
                       (batch.suffix_lens, batch.suffix_tables)):
        for n, row in zip(lens, tabs):
            for j in range(-(-int(n) // B)):
                fill[row[j]] = min(B, int(n) - j * B)
    return LayoutPlan(heads=heads, head_dim=head_dim, block_size=B, dtype=dtype,
                      sm_scale=1.0 / math.sqrt(head_dim), q_scale=1.0,
                      group_ids=batch.group_ids, prefix_lens=batch.prefix_lens,
                      suffix_lens=batch.suffix_lens, prefix_tables=batch.prefix_tables,
                      suffix_tables=batch.suffix_tables, block_fill=fill,
                      poison_block=NB - 1, prefix_parents=batch.prefix_parents)


def test_context_store_batch_end_to_end():
    """Prompts registered in the host context store (a system prompt, three
    task prefixes, own tokens, appended tokens, a prompt that shares nothing)
    produce a batch that the nested entry point decodes to the oracle's result."""
    from paper_2405_19888_amd.context import ContextStore
    say("context store end to end")
    rng = np.random.default_rng(4)
    st = ContextStore(block_size=16, num_blocks=600)
    sysp = rng.integers(0, 1000, size=300).tolist()
    tasks = [rng.integers(0, 1000, size=n).tolist() for n in (50, 77, 120)]
    ctxs = []
    for i in range(12):
        t = tasks[i % 3]
        own = rng.integers(0, 1000, size=int(rng.integers(1, 90))).tolist()
        ctxs.append(st.fill(sysp + t + own, [300, 300 + len(t)]))
    ctxs.append(st.fill(rng.integers(0, 1000, size=40).tolist(), []))
    ctxs.append(st.fill(sysp, [300]))                  # prompt = the system prompt alone
    for c in ctxs[:5]:
        for _ in range(int(rng.integers(1, 20))):
            st.append(c)
    st.append(ctxs[-1])
    batch = st.build_batch(ctxs, pad_block=st.num_blocks)
    assert batch.shape.num_groups == 4 and batch.shape.max_prefix_depth == 2
    plan = plan_from_store(batch, st, heads=8, head_dim=128, dtype="float16")
    data = make_batch(plan, seed=6)
    out, lse = run_gpu(plan, data.to("cuda"))
    assert_close(*to_np(out, lse), *oracle_for(data, plan), "float16", "context store batch")
