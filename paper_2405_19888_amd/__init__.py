"""Shared-prefix decode and prefill attention for AMD MI355X (gfx950).

The compute lives in ``libparrot_attn.so`` (hand-written HIP kernels behind a
C ABI declared in ``include/parrot_attn.h``); this package only builds it and
binds it with ctypes.  Nothing here falls back to a CPU implementation.
"""
from .binding import (  # noqa: F401
    Decoder,
    ParrotError,
    ParrotPrefillRows,
    ParrotProblem,
    ParrotTrace,
    Prefiller,
    load_library,
    make_prefill_rows,
    make_problem,
    parrot_abi_version,
    parrot_hbm_read_ceiling,
    parrot_mfma_issue_ceiling,
    parrot_last_error,
    parrot_nested_prefix_decode,
    parrot_per_request_decode,
    parrot_prefill_single_pass,
    parrot_prefill_workspace_bytes,
    parrot_shared_prefix_decode,
    parrot_shared_prefix_decode_append,
    parrot_shared_prefix_decode_noalloc,
    parrot_shared_prefix_prefill,
    parrot_validate_inputs,
    parrot_validate_nested_inputs,
    parrot_validate_prefill_inputs,
    parrot_workspace_bytes,
    prefill_rows_from_host,
    problem_from_host,
    shared_prefix_decode,
    shared_prefix_prefill,
)
