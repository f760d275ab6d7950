"""Seeded generators for paged decode batches.

Layout of a batch (the paged KV block layout of the library it feeds):
  * K and V pools are [num_blocks, H, B, D] in the batch dtype.  Token t of a
    sequence whose block table row is ``tbl`` lives at pool[tbl[t // B], h,
    t % B, :].
  * Each prefix group g owns a prefix block table row and a prefix length
    P_g >= 1.  Each request r owns a suffix block table row and a suffix length
    S_r >= 0; its group id is g, or -1 when it shares no prefix (then the whole
    context is its suffix).  A request's keys are its group's P_g prefix tokens
    followed by its own S_r suffix tokens.
  * Groups may nest: prefix_parents[g] is the group whose prefix precedes g's
    (-1 for none), always a lower group number.  A request of group g then
    reads the prefixes of g's ancestors, outermost first, then g's, then its
    own tokens.  Flat workloads have every parent -1.
  * Unused token slots of a partly filled block are NaN, and unused block
    table entries point at one all-NaN "poison" block, so any read past a
    length shows up as NaN instead of a plausible number.

Recipe (one plan per workload, shared by all its layers):
  base = numpy default_rng(seed)  (PCG64)
  1. prefix lengths, one per group, then suffix lengths of grouped requests
     (group by group), then ungrouped context lengths;
  2. physical block permutation (identity when the workload is contiguous);
  3. request order permutation (identity when not shuffled).
Values of layer l come from a torch CPU generator seeded with the first
64-bit word (top bit cleared) of numpy's SeedSequence(seed).spawn(L)[l],
drawn in this order:
  q  = N(0,1) * q_scale  as float32, shape [R, H, D]
  K  = N(0,1)            as float32, shape [NB, H, B, D]
  V  = N(0,1)            as float32, shape [NB, H, B, D]
then cast to the workload dtype with round-to-nearest-even.  The device
recipe (``make_device_layers``) draws the same shapes with torch's Philox
generator on the GPU instead; it is used where host generation of many
gigabytes would be too slow, and its values differ from the host recipe.

Prefill queries (``make_prefill_queries``): request r contributes Q_r <= S_r
query rows, its last Q_r own tokens, stacked in request order into a
[sum Q_r, H, D] array; query_offsets[r] is the first row of request r and
query_offsets[R] the row count.  Their values come from a torch CPU generator
seeded with seed * 1000003 + 104729, N(0,1) * q_scale as float32, then cast.
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Optional, Sequence

import numpy as np
import torch

from .configs import ConfigSpec

TORCH_DTYPES = {
    "float32": torch.float32,
    "float16": torch.float16,
    "bfloat16": torch.bfloat16,
}


def _draw_lengths(rng: np.random.Generator, recipe: tuple, n: int) -> np.ndarray:
    kind = recipe[0]
    if n == 0:
        return np.zeros(0, dtype=np.int64)
    if kind == "fixed":
        return np.full(n, int(recipe[1]), dtype=np.int64)
    if kind == "list":
        vals = list(recipe[1])
        if len(vals) != n:
            raise ValueError(f"length list has {len(vals)} entries, need {n}")
        return np.asarray(vals, dtype=np.int64)
    if kind == "uniform":
        a, b = int(recipe[1]), int(recipe[2])
        return rng.integers(a, b, size=n, endpoint=True).astype(np.int64)
    if kind == "lognormal":
        median, sigma, lo, hi = recipe[1:]
        x = rng.lognormal(mean=np.log(median), sigma=sigma, size=n)
        return np.clip(np.round(x), lo, hi).astype(np.int64)
    if kind == "sum_uniform":
        (a1, b1), (a2, b2) = recipe[1], recipe[2]
        x = rng.integers(a1, b1, size=n, endpoint=True)
        y = rng.integers(a2, b2, size=n, endpoint=True)
        return (x + y).astype(np.int64)
    raise ValueError(f"unknown length recipe {recipe!r}")


@dataclass
class LayoutPlan:
    """Lengths, group ids and block tables of one decode batch (no values)."""
    heads: int
    head_dim: int
    block_size: int
    dtype: str
    sm_scale: float
    q_scale: float
    group_ids: np.ndarray        # int32 [R], -1 = no shared prefix
    prefix_lens: np.ndarray      # int32 [NG]
    suffix_lens: np.ndarray      # int32 [R]
    prefix_tables: np.ndarray    # int32 [NG, prefix_stride]
    suffix_tables: np.ndarray    # int32 [R, suffix_stride]
    block_fill: np.ndarray       # int32 [NB] valid token slots per physical block
    poison_block: int            # physical id of the all-NaN block
    prefix_parents: Optional[np.ndarray] = None   # int32 [NG], -1 = outermost

    def __post_init__(self):
        if self.prefix_parents is None:
            self.prefix_parents = np.full(self.num_groups, -1, dtype=np.int32)
        par = np.asarray(self.prefix_parents, dtype=np.int32)
        if par.shape != (self.num_groups,):
            raise ValueError("one parent per group is required")
        if np.any((par >= np.arange(self.num_groups)) | (par < -1)):
            raise ValueError("a group's parent must be -1 or a lower group number")
        self.prefix_parents = par

    @property
    def nested(self) -> bool:
        return bool(np.any(self.prefix_parents >= 0))

    def chain(self, g: int) -> list[int]:
        """Groups whose prefixes a request of group g reads, outermost first."""
        out = []
        while g >= 0:
            out.append(int(g))
            g = int(self.prefix_parents[g])
        return out[::-1]

    def depth(self) -> int:
        """Longest chain of groups (1 for flat groups, 0 without groups)."""
        return max([0] + [len(self.chain(g)) for g in range(self.num_groups)])

    @property
    def num_requests(self) -> int:
        return int(self.group_ids.shape[0])

    @property
    def num_groups(self) -> int:
        return int(self.prefix_lens.shape[0])

    @property
    def num_blocks(self) -> int:
        return int(self.block_fill.shape[0])

    def group_sizes(self) -> list[int]:
        """Requests whose own group is g."""
        return [int((self.group_ids == g).sum()) for g in range(self.num_groups)]

    def reader_counts(self) -> list[int]:
        """Requests that read group g's prefix (g's members and its descendants')."""
        n = [0] * self.num_groups
        for g in self.group_ids:
            for a in self.chain(int(g)):
                n[a] += 1
        return n

    def chain_prefix_len(self, g: int) -> int:
        return int(sum(int(self.prefix_lens[a]) for a in self.chain(g)))

    def context_lens(self) -> np.ndarray:
        """Prefix tokens along the request's chain plus S_r, for every request."""
        p = np.array([self.chain_prefix_len(int(g)) for g in self.group_ids], dtype=np.int64)
        return (p + self.suffix_lens).astype(np.int64)


def build_plan(*, heads: int, head_dim: int, block_size: int, dtype: str,
               group_of_request: Sequence[int], prefix_lens: Sequence[int],
               suffix_lens: Sequence[int], sm_scale: float, q_scale: float = 1.0,
               paged: bool = True, shuffle: bool = False,
               rng: Optional[np.random.Generator] = None,
               prefix_parents: Optional[Sequence[int]] = None) -> LayoutPlan:
    """Allocate blocks and tables for explicit lengths.

    ``group_of_request``, ``suffix_lens`` are in pre-shuffle request order;
    ``prefix_parents`` (default: all -1) nests groups.
    """
    B = int(block_size)
    gor = np.asarray(group_of_request, dtype=np.int64)
    plen = np.asarray(prefix_lens, dtype=np.int64)
    slen = np.asarray(suffix_lens, dtype=np.int64)
    R, NG = gor.shape[0], plen.shape[0]
    if slen.shape[0] != R:
        raise ValueError("one suffix length per request is required")
    if rng is None:
        rng = np.random.default_rng(0)

    # logical block ids: prefix blocks group by group, suffix blocks request by
    # request, then the poison block
    fills: list[int] = []
    pre_logical: list[list[int]] = []
    for g in range(NG):
        n = -(-int(plen[g]) // B)
        pre_logical.append(list(range(len(fills), len(fills) + n)))
        fills += [B] * n
        if n:
            fills[-1] = int(plen[g]) - (n - 1) * B
    suf_logical: list[list[int]] = []
    for r in range(R):
        n = -(-int(slen[r]) // B)
        suf_logical.append(list(range(len(fills), len(fills) + n)))
        fills += [B] * n
        if n:
            fills[-1] = int(slen[r]) - (n - 1) * B
    poison_logical = len(fills)
    fills.append(0)
    NB = len(fills)

    phys = rng.permutation(NB) if paged else np.arange(NB)
    block_fill = np.zeros(NB, dtype=np.int32)
    block_fill[phys] = np.asarray(fills, dtype=np.int32)
    poison = int(phys[poison_logical])

    pstride = max([1] + [len(x) for x in pre_logical])
    sstride = max([1] + [len(x) for x in suf_logical])
    ptab = np.full((NG, pstride), poison, dtype=np.int32)
    for g, blocks in enumerate(pre_logical):
        ptab[g, :len(blocks)] = phys[blocks]
    stab = np.full((R, sstride), poison, dtype=np.int32)
    for r, blocks in enumerate(suf_logical):
        stab[r, :len(blocks)] = phys[blocks]

    order = rng.permutation(R) if shuffle else np.arange(R)
    return LayoutPlan(
        heads=int(heads), head_dim=int(head_dim), block_size=B, dtype=dtype,
        sm_scale=float(sm_scale), q_scale=float(q_scale),
        group_ids=gor[order].astype(np.int32),
        prefix_lens=plen.astype(np.int32),
        suffix_lens=slen[order].astype(np.int32),
        prefix_tables=ptab, suffix_tables=stab[order].copy(),
        block_fill=block_fill, poison_block=poison,
        prefix_parents=None if prefix_parents is None else np.asarray(prefix_parents, np.int32))


def make_plan(cfg: ConfigSpec) -> LayoutPlan:
    rng = np.random.default_rng(cfg.seed)
    NG = cfg.num_groups
    plen = _draw_lengths(rng, cfg.prefix_len, NG)
    n_grouped = sum(cfg.group_sizes)
    slen_grouped = _draw_lengths(rng, cfg.suffix_len, n_grouped)
    slen_ungrouped = _draw_lengths(rng, cfg.ungrouped_len, cfg.ungrouped)
    gor = [g for g, n in enumerate(cfg.group_sizes) for _ in range(n)] + [-1] * cfg.ungrouped
    slen = np.concatenate([slen_grouped, slen_ungrouped])
    return build_plan(heads=cfg.heads, head_dim=cfg.head_dim, block_size=cfg.block_size,
                      dtype=cfg.dtype, group_of_request=gor, prefix_lens=plen,
                      suffix_lens=slen, sm_scale=cfg.sm_scale, q_scale=cfg.q_scale,
                      paged=cfg.paged, shuffle=cfg.shuffle_requests, rng=rng,
                      prefix_parents=cfg.prefix_parents or None)


def flatten_nested(plan: LayoutPlan) -> LayoutPlan:
    """The same batch with one flat group per group that has members: its
    prefix is the concatenation of its chain's prefixes (same physical blocks).

    Only defined when every ancestor prefix fills whole blocks (otherwise the
    concatenated token numbering would not match the block tables).  Used to
    run the flat entry points on a nested workload, as baselines.
    """
    B = plan.block_size
    leaders = [g for g in range(plan.num_groups) if np.any(plan.group_ids == g)]
    for g in leaders:
        for a in plan.chain(g)[:-1]:
            if int(plan.prefix_lens[a]) % B:
                raise ValueError(f"group {a}: prefix length {int(plan.prefix_lens[a])} "
                                 f"is not a multiple of the block size {B}")
    rows, lens = [], []
    for g in leaders:
        row = []
        for a in plan.chain(g):
            n = -(-int(plan.prefix_lens[a]) // B)
            row += [int(x) for x in plan.prefix_tables[a][:n]]
        rows.append(row)
        lens.append(plan.chain_prefix_len(g))
    stride = max([1] + [len(r) for r in rows])
    ptab = np.full((len(leaders), stride), plan.poison_block, dtype=np.int32)
    for i, row in enumerate(rows):
        ptab[i, :len(row)] = row
    remap = {g: i for i, g in enumerate(leaders)}
    gid = np.array([remap.get(int(g), -1) if g >= 0 else -1 for g in plan.group_ids],
                   dtype=np.int32)
    return replace(plan, group_ids=gid, prefix_lens=np.asarray(lens, dtype=np.int32),
                   prefix_tables=ptab, prefix_parents=None)


def one_group_per_request(plan: LayoutPlan) -> LayoutPlan:
    """The same batch with no sharing: every grouped request gets a group of
    its own holding its whole chain of prefixes (same physical blocks, so the
    chain's outer prefixes must fill whole blocks, as for ``flatten_nested``).
    A baseline: the shared-prefix kernels then read each prefix once per
    request."""
    flat = flatten_nested(plan) if plan.nested else plan
    members = [r for r in range(flat.num_requests) if flat.group_ids[r] >= 0]
    src = [int(flat.group_ids[r]) for r in members]
    gid = np.full(flat.num_requests, -1, dtype=np.int32)
    gid[members] = np.arange(len(members), dtype=np.int32)
    ptab = flat.prefix_tables[src] if members else flat.prefix_tables[:0]
    return replace(flat, group_ids=gid, prefix_lens=flat.prefix_lens[src].astype(np.int32),
                   prefix_tables=np.ascontiguousarray(ptab), prefix_parents=None)


@dataclass
class DecodeBatch:
    """One layer of one decode iteration: a plan plus its values (CPU tensors)."""
    plan: LayoutPlan
    q: torch.Tensor          # [R, H, D]
    k_pool: torch.Tensor     # [NB, H, B, D]
    v_pool: torch.Tensor     # [NB, H, B, D]

    @property
    def torch_dtype(self) -> torch.dtype:
        return TORCH_DTYPES[self.plan.dtype]

    def int_arrays(self) -> dict:
        p = self.plan
        return dict(prefix_tables=p.prefix_tables, prefix_lens=p.prefix_lens,
                    suffix_tables=p.suffix_tables, suffix_lens=p.suffix_lens,
                    group_ids=p.group_ids, prefix_parents=p.prefix_parents)

    def to(self, device) -> dict:
        """Tensors of this batch on ``device`` (int arrays as int32 tensors)."""
        out = {k: torch.from_numpy(np.ascontiguousarray(v)).to(device)
               for k, v in self.int_arrays().items()}
        out.update(q=self.q.to(device), k_pool=self.k_pool.to(device),
                   v_pool=self.v_pool.to(device))
        return out


def _nan_slots_mask(plan: LayoutPlan) -> np.ndarray:
    """bool [NB, B]: True where a block slot holds no token."""
    slot = np.arange(plan.block_size)[None, :]
    return slot >= plan.block_fill[:, None]


def _layer_seed(seed: int, layer: int, layers: int) -> int:
    child = np.random.SeedSequence(seed).spawn(layers)[layer]
    return int(child.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


def make_batch(plan: LayoutPlan, layer: int = 0, layers: int = 1, seed: int = 0) -> DecodeBatch:
    """Host-drawn values for layer ``layer`` of ``layers``."""
    g = torch.Generator()
    g.manual_seed(_layer_seed(seed, layer, layers))
    R, H, D, B, NB = plan.num_requests, plan.heads, plan.head_dim, plan.block_size, plan.num_blocks
    q = torch.randn((R, H, D), generator=g, dtype=torch.float32)
    if plan.q_scale != 1.0:
        q.mul_(plan.q_scale)
    k = torch.randn((NB, H, B, D), generator=g, dtype=torch.float32)
    v = torch.randn((NB, H, B, D), generator=g, dtype=torch.float32)
    mask = torch.from_numpy(_nan_slots_mask(plan))[:, None, :, None]
    k.masked_fill_(mask, float("nan"))
    v.masked_fill_(mask, float("nan"))
    td = TORCH_DTYPES[plan.dtype]
    return DecodeBatch(plan=plan, q=q.to(td), k_pool=k.to(td), v_pool=v.to(td))


def make_device_layer(plan: LayoutPlan, layer: int, device, seed: int = 0) -> dict:
    """Device-drawn values of one layer (torch Philox on ``device``).

    Returns q, k_pool, v_pool on ``device`` plus the int arrays as int32
    tensors.  Layer l uses generator seed seed * 1000003 + 7919 * l + 1.
    """
    td = TORCH_DTYPES[plan.dtype]
    R, H, D, B, NB = plan.num_requests, plan.heads, plan.head_dim, plan.block_size, plan.num_blocks
    out = {k: torch.from_numpy(np.ascontiguousarray(v)).to(device)
           for k, v in DecodeBatch(plan, None, None, None).int_arrays().items()}
    mask = torch.from_numpy(_nan_slots_mask(plan)).to(device)[:, None, :, None]
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1_000_003 + 7919 * int(layer) + 1)
    q = torch.randn((R, H, D), generator=g, device=device, dtype=torch.float32)
    if plan.q_scale != 1.0:
        q.mul_(plan.q_scale)
    pools = []
    for _ in range(2):
        x = torch.empty((NB, H, B, D), device=device, dtype=td)
        # draw in slabs to bound the float32 staging buffer
        step = max(1, (1 << 27) // max(1, H * B * D))
        for s in range(0, NB, step):
            e = min(NB, s + step)
            x[s:e] = torch.randn((e - s, H, B, D), generator=g, device=device,
                                 dtype=torch.float32).to(td)
        x.masked_fill_(mask, float("nan"))
        pools.append(x)
    out.update(q=q.to(td), k_pool=pools[0], v_pool=pools[1])
    return out


def make_device_layers(plan: LayoutPlan, layers: int, device, seed: int = 0) -> list[dict]:
    """``make_device_layer`` for layers 0..layers-1."""
    return [make_device_layer(plan, l, device, seed) for l in range(layers)]


def query_offsets_for(plan: LayoutPlan, query_rows: Sequence[int]) -> np.ndarray:
    """int32 [R + 1] row offsets for Q_r = query_rows[r] rows of request r
    (0 <= Q_r <= S_r)."""
    qr = np.asarray(query_rows, dtype=np.int64)
    if qr.shape != (plan.num_requests,):
        raise ValueError("one row count per request")
    if np.any(qr < 0) or np.any(qr > plan.suffix_lens):
        raise ValueError("query rows must lie in [0, S_r]")
    return np.concatenate([[0], np.cumsum(qr)]).astype(np.int32)


def prefill_rows(plan: LayoutPlan, recipe, rng: np.random.Generator) -> np.ndarray:
    """Row counts per request: "all" (Q_r = S_r), an int (min(S_r, n)), or a
    fraction in (0, 1) (ceil(f S_r)); each clipped to [0, S_r]."""
    S = plan.suffix_lens.astype(np.int64)
    if recipe == "all":
        return S.copy()
    if isinstance(recipe, float):
        return np.minimum(S, np.ceil(recipe * S).astype(np.int64))
    return np.minimum(S, int(recipe))


def make_prefill_queries(plan: LayoutPlan, query_rows: Sequence[int], seed: int = 0):
    """(q_rows [sum Q_r, H, D] in the plan dtype, query_offsets int32 [R + 1])."""
    off = query_offsets_for(plan, query_rows)
    g = torch.Generator()
    g.manual_seed(int(seed) * 1_000_003 + 104_729)
    q = torch.randn((int(off[-1]), plan.heads, plan.head_dim), generator=g, dtype=torch.float32)
    if plan.q_scale != 1.0:
        q.mul_(plan.q_scale)
    return q.to(TORCH_DTYPES[plan.dtype]), off


def make_device_prefill_queries(plan: LayoutPlan, query_rows: Sequence[int], device,
                                seed: int = 0, layer: int = 0):
    """Device-drawn prefill rows (torch Philox on ``device``, seed
    seed * 1000003 + 7919 * layer + 104729): (q_rows, offsets as int32 tensor)."""
    off = query_offsets_for(plan, query_rows)
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1_000_003 + 7919 * int(layer) + 104_729)
    q = torch.randn((int(off[-1]), plan.heads, plan.head_dim), generator=g, device=device,
                    dtype=torch.float32)
    if plan.q_scale != 1.0:
        q.mul_(plan.q_scale)
    return q.to(TORCH_DTYPES[plan.dtype]), torch.from_numpy(off).to(device)
