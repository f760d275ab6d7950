"""Full-size parity and coverage probes, in the launch configuration the
benchmark times.

* Every request of the shared-system-prompt (64 x P=6000) and map-reduce
  (4 x 32, LLaMA-13B) workloads, and every request of four layers of the
  32-layer mixed workload (0, 15, 31 and one seeded random layer), on both the
  shared and the per-request path, against the oracle.
* Zero-query probes: with q = 0 every logit is 0, so lse = ln N exactly and
  out = the mean of the request's N values.  N is counted from the lengths and
  the mean from per-block sums of the value pool (a closed form, computed here
  in float64; neither the oracle nor the library is involved).  One key missed
  or counted twice by the prefix chunks or the split-KV pieces moves lse by
  about 1/N, far above the 1e-6 relative bar.
* Spike sweeps: a key planted as c * q with logit 40 takes over its request's
  softmax, so out = that key's value and lse = its logit.  Every request gets
  one spike per call, and the calls walk both sides of every 16-token block
  edge of every prefix and every request's own tokens (prefix positions are
  spread over the group's readers).  Prefix chunks and split-KV runs are whole
  blocks, so every chunk edge and every run boundary the launch uses is pinned
  whatever the chunk size and the run length.

Each case prints its name before touching the GPU.
"""
import math
import sys

import numpy as np
import pytest
import torch

from gpu_util import assert_close, problem_for, run_gpu, run_prefill, to_np
from oracle_pool import oracle_decode, oracle_prefill
from workloads import (get_config, make_batch, make_device_layer, make_device_prefill_queries,
                       make_plan, prefill_rows)

pytestmark = pytest.mark.gpu

B = 16


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def pools_of(d):
    return (d["k_pool"], d["v_pool"], d["k_pool"], d["v_pool"])


# --------------------------------------------------------- closed forms (fp64)
def value_block_sums(v_pool, plan, chunk=256):
    """float64 [NB, H, D]: sum of each physical block's valid token values
    (slots past the block's fill hold NaN and are left out)."""
    NB = plan.num_blocks
    fill = torch.from_numpy(plan.block_fill.astype(np.int64))
    out = torch.zeros((NB, plan.heads, plan.head_dim), dtype=torch.float64)
    slot = torch.arange(B)
    for s in range(0, NB, chunk):
        e = min(NB, s + chunk)
        x = v_pool[s:e].to("cpu", torch.float64)               # [n, H, B, D]
        valid = (slot[None, :] < fill[s:e, None])[:, None, :, None]
        out[s:e] = torch.where(valid, x, torch.zeros((), dtype=torch.float64)).sum(dim=2)
    return out.numpy()


def sequence_blocks(plan, r):
    """Physical blocks of request r's keys: its group chain's prefixes, then
    its own tokens."""
    blocks = []
    for a in (plan.chain(int(plan.group_ids[r])) if plan.group_ids[r] >= 0 else []):
        n = -(-int(plan.prefix_lens[a]) // B)
        blocks += [int(x) for x in plan.prefix_tables[a][:n]]
    n = -(-int(plan.suffix_lens[r]) // B)
    blocks += [int(x) for x in plan.suffix_tables[r][:n]]
    return blocks


def zero_query_expected(plan, v_pool):
    """(mean of the values [R, H, D], ln N [R, H]) for q = 0."""
    sums = value_block_sums(v_pool, plan)
    N = plan.context_lens().astype(np.float64)
    mean = np.stack([sums[sequence_blocks(plan, r)].sum(axis=0) / N[r]
                     for r in range(plan.num_requests)])
    return mean, np.repeat(np.log(N)[:, None], plan.heads, axis=1)


def check_zero_query(plan, o, l, mean, ln_n, what):
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(l)), what
    lerr = np.max(np.abs(l - ln_n) / ln_n)
    assert lerr < 1e-6, f"{what}: lse vs ln N rel err {lerr:.3e}"
    # the mean is exact in fp32 up to a few ulps of the partial sums; the
    # output's rounding to the cache type (half an ulp) dominates
    half_ulp = 2.0 ** -8 if plan.dtype == "bfloat16" else 2.0 ** -11
    bound = half_ulp * np.maximum(np.abs(mean), 2.0 ** -6) + 2e-5
    worst = np.max(np.abs(o - mean) - bound)
    assert worst <= 0, f"{what}: out vs mean of V exceeds its bound by {worst:.3e}"


# --------------------------------------------------------------- spike sweeps
def edge_positions(n):
    """Both sides of every block edge of an n-token sequence, plus its first
    and last token."""
    pos = {0, n - 1}
    for b in range(1, -(-n // B)):
        pos |= {B * b - 1, B * b}
    return sorted(p for p in pos if 0 <= p < n)


def spike_queues(plan):
    """Per request, the (sequence, token) positions to spike, one per call:
    prefix positions of every group spread round-robin over its readers, then
    the request's own edge positions."""
    R = plan.num_requests
    queues = [[] for _ in range(R)]
    readers = [[] for _ in range(plan.num_groups)]
    for r in range(R):
        if plan.group_ids[r] >= 0:
            for a in plan.chain(int(plan.group_ids[r])):
                readers[a].append(r)
    for g in range(plan.num_groups):
        if not readers[g]:
            continue
        for i, t in enumerate(edge_positions(int(plan.prefix_lens[g]))):
            queues[readers[g][i % len(readers[g])]].append(("prefix", g, t))
    for r in range(R):
        for t in edge_positions(int(plan.suffix_lens[r])):
            queues[r].append(("own", r, t))
    return queues


def spike_sweep(plan, dev, what, paths=(True, False), max_calls=None):
    """Run the spike calls on `dev` (device pools are modified and restored
    call by call) and check every spiked request on each path."""
    q = dev["q"].to("cpu", torch.float64)                       # [R, H, D]
    qq = (q * q).sum(-1)                                        # [R, H]
    c = 40.0 / (plan.sm_scale * qq)
    keys = (c[..., None] * q).to(dev["k_pool"].dtype)           # the spike key of (r, h)
    logit = (plan.sm_scale * (q * keys.double()).sum(-1)).numpy()
    queues = spike_queues(plan)
    calls = max(len(x) for x in queues)
    if max_calls is not None:
        calls = min(calls, max_calls)
    prob = problem_for(plan)
    from paper_2405_19888_amd import Decoder
    decs = {p: Decoder(prob) for p in paths}
    k_dev = dev["k_pool"]
    checked = 0
    for i in range(calls):
        reqs, blks, slots = [], [], []
        for r, qu in enumerate(queues):
            if i >= len(qu):
                continue
            kind, s, t = qu[i]
            row = plan.prefix_tables[s] if kind == "prefix" else plan.suffix_tables[s]
            reqs.append(r); blks.append(int(row[t // B])); slots.append(t % B)
        bi = torch.tensor(blks, device="cuda"); si = torch.tensor(slots, device="cuda")
        ri = torch.tensor(reqs)
        saved = k_dev[bi, :, si].clone()
        k_dev[bi, :, si] = keys[ri].to("cuda")
        v = dev["v_pool"][bi, :, si].to("cpu", torch.float64).numpy()       # [n, H, D]
        try:
            for shared in paths:
                out, lse = decs[shared](dev, shared=shared, nested=plan.nested)
                o, l = to_np(out[ri.to("cuda")], lse[ri.to("cuda")])
                tol = 1e-3 * np.maximum(1.0, np.abs(v).max(axis=(1, 2)))
                err = np.abs(o - v).max(axis=(1, 2))
                bad = np.nonzero(err > tol)[0]
                assert bad.size == 0, (f"{what} call {i} shared={shared}: request {reqs[bad[0]]} "
                                       f"spike {queues[reqs[bad[0]]][i]} out err {err[bad[0]]:.3e}")
                s = logit[reqs]
                lerr = np.abs(l - s) / np.abs(s)
                assert lerr.max() < 1e-5, (f"{what} call {i} shared={shared}: lse rel err "
                                           f"{lerr.max():.3e}")
        finally:
            k_dev[bi, :, si] = saved
        checked += len(reqs)
        if (i + 1) % 100 == 0:
            say(what, "spike call", i + 1, "of", calls)
    torch.cuda.synchronize()
    return calls, checked


# ------------------------------------------------------- every request, C3/C4
@pytest.mark.parametrize("name", ["c3", "c4"])
def test_every_request_matches_oracle(name):
    cfg = get_config(name)
    plan = make_plan(cfg)
    say(name, cfg.name, "every request, both paths")
    batch = make_batch(plan)
    dev = batch.to("cuda")
    res = {s: to_np(*run_gpu(plan, dev, shared=s)) for s in (True, False)}
    say(name, "oracle on", plan.num_requests, "requests")
    ref = oracle_decode(batch.q, (batch.k_pool, batch.v_pool, batch.k_pool, batch.v_pool), plan)
    for shared, (o, l) in res.items():
        assert_close(o, l, *ref, plan.dtype, f"{cfg.name} every request shared={shared}")
    # extra: the two GPU paths agree with each other within the same bar
    (o1, l1), (o2, l2) = res[True], res[False]
    assert np.max(np.abs(o1 - o2)) <= 2e-3
    assert np.max(np.abs(l1 - l2) / np.maximum(1, np.abs(l2))) <= 1e-4


# ---------------------------------------------------- 32-layer mixed workload
def _checked_layers(n_layers):
    rng = np.random.default_rng(0)
    rest = [l for l in range(n_layers) if l not in (0, 15, 31)]
    return [0, 15, 31, int(rng.choice(rest))]


C5_LAYERS = _checked_layers(32)


@pytest.fixture(scope="module")
def mixed_workload():
    """All 32 layers resident on the device (about 4 GB of bf16 KV each);
    every layer decoded on both paths; the outputs of the checked layers kept,
    with those layers' inputs."""
    cfg = get_config("c5")
    plan = make_plan(cfg)
    say(cfg.name, "layers", cfg.layers, "blocks", plan.num_blocks, "checked", C5_LAYERS)
    from paper_2405_19888_amd import Decoder
    dec = Decoder(problem_for(plan))
    kept, outs = {}, {}
    layers = []
    for l in range(cfg.layers):
        layers.append(make_device_layer(plan, l, "cuda", seed=cfg.seed))
        if l % 8 == 7:
            say(cfg.name, "layers resident:", l + 1)
    run_gpu(plan, layers[0], decoder=dec)            # validates the inputs once
    for shared in (True, False):
        for l, dev in enumerate(layers):
            out, lse = dec(dev, shared=shared)
            if l in C5_LAYERS:
                outs[(l, shared)] = (out.clone(), lse.clone())
    torch.cuda.synchronize()
    for l in C5_LAYERS:
        kept[l] = layers[l]
    del layers
    yield plan, kept, outs
    kept.clear(); outs.clear()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("layer", C5_LAYERS)
def test_mixed_32_layer_every_request(mixed_workload, layer):
    plan, kept, outs = mixed_workload
    dev = kept[layer]
    say("mixed_7b_32layer layer", layer, "oracle on", plan.num_requests, "requests")
    ref = oracle_decode(dev["q"], pools_of(dev), plan)
    for shared in (True, False):
        o, l = to_np(*outs[(layer, shared)])
        assert_close(o, l, *ref, plan.dtype, f"layer {layer} every request shared={shared}")


# ------------------------------------------------------- zero-query, decode
ZERO_QUERY_DECODE = ["c2", "c3", "c4", "c5", "nested"]


@pytest.mark.parametrize("name", ZERO_QUERY_DECODE)
def test_zero_query_full_size(name):
    cfg = get_config(name)
    plan = make_plan(cfg)
    say("zero-query full size", cfg.name)
    dev = make_device_layer(plan, 0, "cuda", seed=cfg.seed)
    dev["q"].zero_()
    mean, ln_n = zero_query_expected(plan, dev["v_pool"])
    for shared in ((True,) if plan.nested else (True, False)):
        o, l = to_np(*run_gpu(plan, dev, shared=shared))
        check_zero_query(plan, o, l, mean, ln_n, f"{cfg.name} shared={shared}")


# ------------------------------------------------------------- spike sweeps
@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5", "nested"])
def test_spike_sweep_full_size(name):
    cfg = get_config(name)
    plan = make_plan(cfg)
    dev = make_device_layer(plan, 0, "cuda", seed=cfg.seed)
    say("spike sweep full size", cfg.name)
    run_gpu(plan, dev)                                   # validates the inputs
    paths = (True,) if plan.nested else (True, False)
    calls, checked = spike_sweep(plan, dev, cfg.name, paths=paths)
    say(cfg.name, "spike calls", calls, "spiked requests checked", checked)
    # every request had at least its own first and last token spiked
    assert checked >= sum(min(2, int(s)) for s in plan.suffix_lens)


# ----------------------------------------------------- zero-query, prefill
def zero_query_prefill_expected(plan, v_pool, off):
    """(mean of the visible values [T, H, D], ln N [T, H]) for q = 0: row j of
    request r sits at own position p = S_r - Q_r + j and sees the chain's
    prefix tokens plus own tokens 0..p."""
    sums = value_block_sums(v_pool, plan)
    T = int(off[-1])
    H, D = plan.heads, plan.head_dim
    mean = np.zeros((T, H, D))
    n_keys = np.zeros(T)
    for r in range(plan.num_requests):
        a, b = int(off[r]), int(off[r + 1])
        if b == a:
            continue
        g = int(plan.group_ids[r])
        pre_blocks = []
        P = 0
        for x in (plan.chain(g) if g >= 0 else []):
            n = -(-int(plan.prefix_lens[x]) // B)
            pre_blocks += [int(y) for y in plan.prefix_tables[x][:n]]
            P += int(plan.prefix_lens[x])
        pre_sum = sums[pre_blocks].sum(axis=0) if pre_blocks else np.zeros((H, D))
        S = int(plan.suffix_lens[r])
        nb = -(-S // B)
        own = v_pool[torch.as_tensor(plan.suffix_tables[r][:nb].astype(np.int64),
                                     device=v_pool.device)]
        own = own.to("cpu", torch.float64).permute(0, 2, 1, 3).reshape(nb * B, H, D)[:S]
        cum = torch.cumsum(own, dim=0).numpy()                      # [S, H, D]
        p = np.arange(S - (b - a), S)
        n = P + p + 1
        mean[a:b] = (pre_sum[None] + cum[p]) / n[:, None, None]
        n_keys[a:b] = n
    return mean, np.repeat(np.log(n_keys)[:, None], H, axis=1)


@pytest.mark.parametrize("name", ["prefill", "prefill_q16"])
def test_prefill_zero_query_full_size(name, monkeypatch):
    """The benchmark's prefill workloads in the plan the benchmark times."""
    monkeypatch.delenv("PARROT_PREFILL_SINGLE_PASS", raising=False)
    cfg = get_config(name)
    plan = make_plan(cfg)
    qr = prefill_rows(plan, cfg.prefill_rows, None)
    say("prefill zero-query full size", cfg.name, int(qr.sum()), "rows")
    dev = make_device_layer(plan, 0, "cuda", seed=cfg.seed)
    dev["q_rows"], dev["query_offsets"] = make_device_prefill_queries(plan, qr, "cuda", cfg.seed, 0)
    dev["q_rows"].zero_()
    off = dev["query_offsets"].cpu().numpy()
    o, l = to_np(*run_prefill(plan, dev, off))
    mean, ln_n = zero_query_prefill_expected(plan, dev["v_pool"], off)
    check_zero_query(plan, o, l, mean, ln_n, f"{cfg.name} zero query")


# ------------------------------------------------ prefill, many rows vs oracle
@pytest.mark.parametrize("name", ["prefill", "prefill_q16"])
def test_prefill_tile_edge_rows_match_oracle(name, monkeypatch):
    """Rows at every 128-row tile edge, every request's first and last row,
    and all rows of the request with the fewest rows, against the oracle, in
    the plan the benchmark times."""
    monkeypatch.delenv("PARROT_PREFILL_SINGLE_PASS", raising=False)
    cfg = get_config(name)
    plan = make_plan(cfg)
    qr = prefill_rows(plan, cfg.prefill_rows, None)
    dev = make_device_layer(plan, 0, "cuda", seed=cfg.seed)
    dev["q_rows"], dev["query_offsets"] = make_device_prefill_queries(plan, qr, "cuda", cfg.seed, 0)
    off = dev["query_offsets"].cpu().numpy()
    T = int(off[-1])
    rows = {t for t in range(T) if t % 128 in (0, 127)}
    for r in range(plan.num_requests):
        if off[r + 1] > off[r]:
            rows |= {int(off[r]), int(off[r + 1]) - 1}
    nz = [r for r in range(plan.num_requests) if off[r + 1] > off[r]]
    r = min(nz, key=lambda x: off[x + 1] - off[x])
    rows |= set(range(int(off[r]), int(off[r + 1])))
    rows = sorted(rows)
    say("prefill rows vs oracle", cfg.name, len(rows), "of", T, "rows")
    o, l = to_np(*run_prefill(plan, dev, off))
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(l))
    ref = oracle_prefill(dev["q_rows"], off, pools_of(dev), plan, rows=rows)
    assert_close(o[rows], l[rows], *ref, plan.dtype, f"{cfg.name} tile-edge rows")
