"""The seeded input generators (CPU only)."""
import numpy as np
import pytest
import torch

from workloads import build_plan, get_config, make_batch, make_plan, zipf_group_sizes
from workloads.configs import ALIASES


def test_zipf_split():
    assert zipf_group_sizes(256, 8, 1.1) == [102, 48, 31, 22, 17, 14, 12, 10]
    assert sum(zipf_group_sizes(1000, 7, 0.8)) == 1000


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_plan_shapes_and_ranges(name):
    cfg = get_config(name)
    p = make_plan(cfg)
    assert p.num_requests == cfg.num_requests
    assert p.group_sizes() == list(cfg.group_sizes)
    assert int((p.group_ids == -1).sum()) == cfg.ungrouped
    grouped = p.group_ids >= 0
    s = p.suffix_lens[grouped]
    kind = cfg.suffix_len[0]
    if kind == "uniform":
        assert s.min() >= cfg.suffix_len[1] and s.max() <= cfg.suffix_len[2]
    if kind == "lognormal":
        assert s.min() >= cfg.suffix_len[3] and s.max() <= cfg.suffix_len[4]
    if kind == "list":
        assert list(s) == list(cfg.suffix_len[1])
    if cfg.prefix_len[0] == "uniform":
        assert p.prefix_lens.min() >= cfg.prefix_len[1] and p.prefix_lens.max() <= cfg.prefix_len[2]
    if cfg.ungrouped:
        u = p.suffix_lens[~grouped]
        lo = cfg.ungrouped_len[1][0] + cfg.ungrouped_len[2][0]
        hi = cfg.ungrouped_len[1][1] + cfg.ungrouped_len[2][1]
        assert u.min() >= lo and u.max() <= hi


@pytest.mark.parametrize("name", ["c1", "c2", "c4", "c5"])
def test_every_block_used_once(name):
    p = make_plan(get_config(name))
    B = p.block_size
    used = []
    for g in range(p.num_groups):
        used += list(p.prefix_tables[g][: -(-int(p.prefix_lens[g]) // B)])
    for r in range(p.num_requests):
        used += list(p.suffix_tables[r][: -(-int(p.suffix_lens[r]) // B)])
    used.append(p.poison_block)
    assert sorted(used) == list(range(p.num_blocks))
    # table padding points at the poison block only
    for g in range(p.num_groups):
        assert np.all(p.prefix_tables[g][-(-int(p.prefix_lens[g]) // B):] == p.poison_block)
    # the fill of each block matches the lengths
    assert int(p.block_fill.sum()) == int(p.prefix_lens.sum() + p.suffix_lens.sum())


def test_contiguous_tables_are_identity():
    p = make_plan(get_config("c1"))
    assert list(p.prefix_tables[0]) == list(range(8))
    assert list(p.suffix_tables[:, 0]) == [8, 9, 11, 13]   # S = 16, 24, 32, 20
    assert list(p.group_ids) == [0, 0, 0, 0]


def test_values_deterministic_and_poisoned():
    p = make_plan(get_config("c1"))
    a, b = make_batch(p), make_batch(p)
    assert torch.equal(a.q, b.q)
    assert torch.equal(torch.nan_to_num(a.k_pool), torch.nan_to_num(b.k_pool))
    # partial-block slots and the poison block hold NaN; every token slot is finite
    for blk in range(p.num_blocks):
        f = int(p.block_fill[blk])
        assert torch.isfinite(a.k_pool[blk, :, :f]).all()
        assert torch.isnan(a.v_pool[blk, :, f:]).all()
    other = make_batch(p, seed=1)
    assert not torch.equal(a.q, other.q)


def test_layers_differ():
    p = make_plan(get_config("c1"))
    l0, l1 = make_batch(p, 0, 2), make_batch(p, 1, 2)
    assert not torch.equal(l0.q, l1.q)


def test_dtype_cast_is_round_to_nearest_even():
    rng = np.random.default_rng(0)
    plan = build_plan(heads=1, head_dim=8, block_size=16, dtype="bfloat16",
                      group_of_request=[0], prefix_lens=[3], suffix_lens=[2],
                      sm_scale=1.0, rng=rng)
    b = make_batch(plan)
    assert b.k_pool.dtype == torch.bfloat16 and b.q.dtype == torch.bfloat16


def test_aliases_cover_all_configs():
    assert sorted(ALIASES.values()) == sorted(["tiny", "llama7b_g32_p2048", "sysprompt_g64_p6000",
                                               "mapreduce_13b_4x32", "mixed_7b_32layer",
                                               "nested_sys6000_8x8_fs256", "prefill_sys6000_g64",
                                               "prefill_sys6000_g64_q16"])
    from workloads import CONFIGS
    assert set(ALIASES.values()) == set(CONFIGS)


def test_nested_plan_chains_and_flattening():
    from workloads.gen import flatten_nested
    plan = make_plan(get_config("nested"))
    assert plan.depth() == 2 and plan.nested
    assert plan.reader_counts() == [64] + [8] * 8
    for r in range(plan.num_requests):
        g = int(plan.group_ids[r])
        assert plan.chain(g) == [0, g] and g >= 1
        assert plan.context_lens()[r] == 6000 + 256 + plan.suffix_lens[r]
    flat = flatten_nested(plan)
    assert not flat.nested and flat.num_groups == 8
    assert np.array_equal(flat.context_lens(), plan.context_lens())
    # the flat prefix of a request's group is its chain's blocks in order
    B = plan.block_size
    for r in range(plan.num_requests):
        g, fg = int(plan.group_ids[r]), int(flat.group_ids[r])
        want = list(plan.prefix_tables[0][:6000 // B]) + list(plan.prefix_tables[g][:256 // B])
        assert list(flat.prefix_tables[fg][:len(want)]) == want


def test_parents_must_point_to_lower_groups():
    with pytest.raises(ValueError):
        build_plan(heads=1, head_dim=64, block_size=16, dtype="float32", group_of_request=[0, 1],
                   prefix_lens=[16, 16], suffix_lens=[1, 1], sm_scale=1.0,
                   prefix_parents=[1, -1])


def test_prefill_queries_layout():
    from workloads import make_prefill_queries, prefill_rows, query_offsets_for
    plan = make_plan(get_config("tiny"))
    rng = np.random.default_rng(0)
    for recipe in ("all", 3, 0.5):
        qr = prefill_rows(plan, recipe, rng)
        assert np.all(qr >= 0) and np.all(qr <= plan.suffix_lens)
        q, off = make_prefill_queries(plan, qr, seed=2)
        assert off[0] == 0 and off[-1] == q.shape[0] == qr.sum()
        assert np.array_equal(np.diff(off), qr)
        assert q.shape[1:] == (plan.heads, plan.head_dim)
        q2, _ = make_prefill_queries(plan, qr, seed=2)
        assert torch.equal(q, q2)
    with pytest.raises(ValueError):
        query_offsets_for(plan, plan.suffix_lens + 1)
    with pytest.raises(ValueError):
        query_offsets_for(plan, [1])
