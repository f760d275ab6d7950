"""Shared-prefix decode attention for AMD MI355X (gfx950).

The compute lives in ``libparrot_attn.so`` (hand-written HIP kernels behind a
C ABI declared in ``include/parrot_attn.h``); this package only builds it and
binds it with ctypes.  Nothing here falls back to a CPU implementation.
"""
from .binding import (  # noqa: F401
    Decoder,
    ParrotError,
    ParrotProblem,
    ParrotTrace,
    load_library,
    make_problem,
    parrot_abi_version,
    parrot_last_error,
    parrot_nested_prefix_decode,
    parrot_per_request_decode,
    parrot_shared_prefix_decode,
    parrot_shared_prefix_decode_append,
    parrot_validate_inputs,
    parrot_validate_nested_inputs,
    parrot_workspace_bytes,
    problem_from_host,
)
