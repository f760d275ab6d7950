"""Seeded synthetic decode batches for shared-prefix decode attention.

This package only draws inputs: lengths, block tables, group ids and the
random query / key / value values.  It holds none of the attention
arithmetic, so that the CPU oracle (``oracle/``) and the HIP library
(``paper_2405_19888_amd``) can both be fed from it without sharing code.
"""
from .configs import CONFIGS, ConfigSpec, get_config, zipf_group_sizes
from .gen import DecodeBatch, LayoutPlan, build_plan, make_plan, make_batch, make_device_layer, make_device_layers
from .gen import (make_device_prefill_queries, make_prefill_queries, one_group_per_request,
                  prefill_rows, query_offsets_for)

__all__ = [
    "CONFIGS", "ConfigSpec", "get_config", "zipf_group_sizes",
    "DecodeBatch", "LayoutPlan", "build_plan", "make_plan", "make_batch", "make_device_layer", "make_device_layers",
    "make_prefill_queries", "prefill_rows", "query_offsets_for", "make_device_prefill_queries",
    "one_group_per_request",
]
