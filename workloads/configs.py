"""The five synthetic decode workloads, a nested one, two prefill workloads,
plus the prefix-length sweep.

Each workload is one continuous-batching decode iteration (one query per
request) over a paged KV cache, shaped after the model sizes and sharing
patterns the paper evaluates (Section 8.1 testbed and models; Section 8.3
shared system prompt; Table 2 on which workloads share prompts).  None of the
paper's datasets or prompts are used: every value is a seeded normal draw.

Length recipes, in this module's notation:
  ("fixed", v)                 every draw is v
  ("list", [v0, v1, ...])      the i-th draw is v_i
  ("uniform", a, b)            integers uniform on [a, b], both ends included
  ("lognormal", median, sigma, lo, hi)
                               exp(N(ln median, sigma)), rounded half-to-even,
                               then clipped to [lo, hi]
  ("sum_uniform", (a1, b1), (a2, b2))
                               sum of two independent uniform integer draws
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Sequence


def zipf_group_sizes(total: int, groups: int, s: float) -> list[int]:
    """Split ``total`` requests over ``groups`` groups with Zipf(s) shares.

    Shares are proportional to k**-s for k = 1..groups; the integer split is
    the largest-remainder method (floors first, then one extra request to the
    groups with the largest fractional parts, ties to the lower k).
    """
    w = [k ** -s for k in range(1, groups + 1)]
    tot = sum(w)
    raw = [total * x / tot for x in w]
    base = [math.floor(x) for x in raw]
    left = total - sum(base)
    order = sorted(range(groups), key=lambda i: (-(raw[i] - base[i]), i))
    for i in order[:left]:
        base[i] += 1
    return base


@dataclass(frozen=True)
class ConfigSpec:
    name: str
    description: str
    layers: int
    heads: int
    head_dim: int
    block_size: int
    dtype: str                      # "float32" | "float16" | "bfloat16"
    group_sizes: tuple              # requests whose own group is g
    prefix_len: tuple               # length recipe, one draw per group
    suffix_len: tuple               # length recipe, one draw per grouped request
    prefix_parents: tuple = ()      # parent group per group (-1 = none); () = flat
    ungrouped: int = 0              # requests with no shared prefix
    ungrouped_len: tuple = ("fixed", 0)   # whole-context length recipe for them
    q_scale: float = 1.0            # q is drawn N(0,1) * q_scale
    sm_scale: float = 1.0           # logits = sm_scale * q.k
    paged: bool = True              # False: identity block tables (contiguous KV)
    shuffle_requests: bool = True   # interleave group members in the batch
    seed: int = 0
    prefill_rows: object = None     # prefill workloads: rows per request ("all", n or a
                                    # fraction of S_r; see gen.prefill_rows); None = decode

    @property
    def num_requests(self) -> int:
        return sum(self.group_sizes) + self.ungrouped

    @property
    def num_groups(self) -> int:
        return len(self.group_sizes)

    def with_(self, **kw) -> "ConfigSpec":
        return replace(self, **kw)


_INV_SQRT128 = 1.0 / math.sqrt(128.0)

CONFIGS: dict[str, ConfigSpec] = {
    "tiny": ConfigSpec(
        name="tiny",
        description="1 layer, 1 group of 4, 4 heads x 64, prefix 128, suffix "
                    "{16,24,32,20}, fp32, q pre-scaled by 1/8, contiguous KV",
        layers=1, heads=4, head_dim=64, block_size=16, dtype="float32",
        group_sizes=(4,), prefix_len=("fixed", 128),
        suffix_len=("list", [16, 24, 32, 20]),
        q_scale=1.0 / 8.0, sm_scale=1.0, paged=False, shuffle_requests=False),
    "llama7b_g32_p2048": ConfigSpec(
        name="llama7b_g32_p2048",
        description="LLaMA-7B layer: 32 heads x 128, fp16 paged (B=16), "
                    "1 group of 32, prefix 2048, suffix U[64,512]",
        layers=1, heads=32, head_dim=128, block_size=16, dtype="float16",
        group_sizes=(32,), prefix_len=("fixed", 2048),
        suffix_len=("uniform", 64, 512), sm_scale=_INV_SQRT128),
    "sysprompt_g64_p6000": ConfigSpec(
        name="sysprompt_g64_p6000",
        description="long shared system prompt: 32 heads x 128, fp16 paged, "
                    "1 group of 64, prefix 6000, suffix U[100,1000]",
        layers=1, heads=32, head_dim=128, block_size=16, dtype="float16",
        group_sizes=(64,), prefix_len=("fixed", 6000),
        suffix_len=("uniform", 100, 1000), sm_scale=_INV_SQRT128),
    "mapreduce_13b_4x32": ConfigSpec(
        name="mapreduce_13b_4x32",
        description="LLaMA-13B layer: 40 heads x 128, fp16 paged, 4 groups of "
                    "32 with prefixes 1024/2048/3072/4096, suffix "
                    "lognormal(median 256, sigma 1) clipped to [16,2048]",
        layers=1, heads=40, head_dim=128, block_size=16, dtype="float16",
        group_sizes=(32, 32, 32, 32),
        prefix_len=("list", [1024, 2048, 3072, 4096]),
        suffix_len=("lognormal", 256.0, 1.0, 16, 2048), sm_scale=_INV_SQRT128),
    "mixed_7b_32layer": ConfigSpec(
        name="mixed_7b_32layer",
        description="LLaMA-7B full depth: 32 layers x 32 heads x 128, bf16 "
                    "paged, 256 requests in 8 Zipf(1.1) groups, prefix "
                    "U[512,4096], suffix U[32,1024], plus 32 ungrouped "
                    "requests with context U[512,4096]+U[32,1024]",
        layers=32, heads=32, head_dim=128, block_size=16, dtype="bfloat16",
        group_sizes=tuple(zipf_group_sizes(256, 8, 1.1)),
        prefix_len=("uniform", 512, 4096), suffix_len=("uniform", 32, 1024),
        ungrouped=32, ungrouped_len=("sum_uniform", (512, 4096), (32, 1024)),
        sm_scale=_INV_SQRT128),
    "nested_sys6000_8x8_fs256": ConfigSpec(
        name="nested_sys6000_8x8_fs256",
        description="two-level sharing, LLaMA-7B layer: 32 heads x 128, fp16 "
                    "paged; a 6000-token system prompt (group 0) shared by 8 "
                    "sub-groups, each adding a 256-token few-shot block and "
                    "holding 8 requests; own tokens U[64,512]",
        layers=1, heads=32, head_dim=128, block_size=16, dtype="float16",
        group_sizes=(0,) + (8,) * 8, prefix_parents=(-1,) + (0,) * 8,
        prefix_len=("list", [6000] + [256] * 8),
        suffix_len=("uniform", 64, 512), sm_scale=_INV_SQRT128),
    "prefill_sys6000_g64": ConfigSpec(
        name="prefill_sys6000_g64",
        description="Fill of 64 contexts forked from a 6000-token system prompt, "
                    "LLaMA-7B layer: 32 heads x 128, fp16 paged; each fills its "
                    "own prompt of U[100,1000] tokens (every own token a query row)",
        layers=1, heads=32, head_dim=128, block_size=16, dtype="float16",
        group_sizes=(64,), prefix_len=("fixed", 6000),
        suffix_len=("uniform", 100, 1000), sm_scale=_INV_SQRT128, prefill_rows="all"),
    "prefill_sys6000_g64_q16": ConfigSpec(
        name="prefill_sys6000_g64_q16",
        description="as prefill_sys6000_g64, but each context fills only its last "
                    "16 own tokens (a continued, chunked prompt)",
        layers=1, heads=32, head_dim=128, block_size=16, dtype="float16",
        group_sizes=(64,), prefix_len=("fixed", 6000),
        suffix_len=("uniform", 100, 1000), sm_scale=_INV_SQRT128, prefill_rows=16),
}

# Short aliases in the order the workloads are listed (C1..C5).
ALIASES = {
    "c1": "tiny", "c2": "llama7b_g32_p2048", "c3": "sysprompt_g64_p6000",
    "c4": "mapreduce_13b_4x32", "c5": "mixed_7b_32layer",
    "nested": "nested_sys6000_8x8_fs256",
    "prefill": "prefill_sys6000_g64", "prefill_q16": "prefill_sys6000_g64_q16",
}


def get_config(name: str, **overrides) -> ConfigSpec:
    if name.startswith("sweep_p"):
        cfg = prefix_sweep(int(name[len("sweep_p"):]))
        return cfg.with_(**overrides) if overrides else cfg
    cfg = CONFIGS[ALIASES.get(name, name)]
    return cfg.with_(**overrides) if overrides else cfg


def prefix_sweep(prefix_len: int) -> ConfigSpec:
    """The LLaMA-7B one-group shape with a chosen shared-prefix length."""
    base = CONFIGS["llama7b_g32_p2048"]
    return base.with_(name=f"sweep_p{prefix_len}", prefix_len=("fixed", prefix_len))


SWEEP_PREFIX_LENS: Sequence[int] = (256, 512, 1024, 2048, 4096, 8192, 16384)
