"""CPU oracle for shared-prefix decode attention -- TEST INFRASTRUCTURE ONLY.

This package is test infrastructure, not the product.  Only the test suite, the smoke
check of the entry module and the CPU-baseline leg of the benchmark may import
it; the library path never calls it and has no CPU fallback.

What it computes (Section 5.3, "Sharing Prompt Prefix", and Section 7,
"Kernel Optimization"): decode-phase softmax attention of one query per request
over that request's whole context, i.e. the shared prefix of its group followed
by its own non-shared tokens (or, with nested groups, the prefixes of the
group's ancestors first), with keys and values read from a paged KV cache
through block tables.  The paper's two-stage kernel reaches exactly this result
(up to rounding order), so the oracle is the plain definition written out, in
float64, per request and per head, with no blocking, splitting or fusion.
The prefill of a forked context (Section 7, Fill with a parent context) is the
same definition per new token, with each request's own tokens cut after the
token's position (causal).

Pinning (the tests hold the pins): brute force in pure-Python loops on tiny
inputs, a hand-computed worked example, torch's scaled_dot_product_attention
in float64 on contiguous input, closed forms (zero query, single key,
identical keys, a dominant "spike" key), softmax weights that sum to one,
invariance under physical block permutation, and the prefix/suffix
decomposition identity; for prefill, pure-Python brute force, masked
scaled_dot_product_attention in float64, the last row equal to a decode step,
causality (later own tokens change nothing) and a single-key first row.  Every
function here is pinned by at least one of them.
"""
from .attention import (
    to_f64,
    gather_sequence,
    attend,
    merge_segments,
    softmax_weights,
    group_chain,
    request_kv,
    shared_prefix_decode,
    prefill_positions,
    shared_prefix_prefill,
)

__all__ = [
    "to_f64", "gather_sequence", "attend", "merge_segments", "softmax_weights",
    "group_chain", "request_kv", "shared_prefix_decode",
    "prefill_positions", "shared_prefix_prefill",
]
