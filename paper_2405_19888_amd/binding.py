"""ctypes binding of libparrot_attn (argument marshalling only).

Every function here forwards to the C entry point of the same name in
``include/parrot_attn.h``; torch tensors are passed as raw device pointers and
the stream as torch's current HIP stream.  There is no fallback: if the shared
library is missing or a call fails, an exception says so.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libparrot_attn.so")

PARROT_OK = 0
PARROT_ERR_INVALID_ARGUMENT = 1
PARROT_ERR_UNSUPPORTED = 2
PARROT_ERR_WORKSPACE_TOO_SMALL = 3
PARROT_ERR_HIP = 4

DTYPE_CODES = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}


class ParrotError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libparrot_attn status {status}: {msg}")
        self.status = status


class ParrotProblem(ctypes.Structure):
    _fields_ = [
        ("num_requests", ctypes.c_int32),
        ("num_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("num_groups", ctypes.c_int32),
        ("max_group_size", ctypes.c_int32),
        ("max_prefix_len", ctypes.c_int32),
        ("max_suffix_len", ctypes.c_int32),
        ("prefix_table_stride", ctypes.c_int32),
        ("suffix_table_stride", ctypes.c_int32),
        ("num_prefix_blocks", ctypes.c_int32),
        ("num_suffix_blocks", ctypes.c_int32),
        ("dtype", ctypes.c_int),
        ("sm_scale", ctypes.c_float),
        ("max_prefix_depth", ctypes.c_int32),
    ]


class ParrotTrace(ctypes.Structure):
    _fields_ = [
        ("partials_start", ctypes.c_void_p),
        ("partials_stop", ctypes.c_void_p),
        ("merge_start", ctypes.c_void_p),
        ("merge_stop", ctypes.c_void_p),
    ]


class ParrotPrefillRows(ctypes.Structure):
    _fields_ = [
        ("num_query_rows", ctypes.c_int32),
        ("max_query_rows", ctypes.c_int32),
        ("max_group_rows", ctypes.c_int32),
    ]


EXPORTED = (
    "parrot_workspace_bytes", "parrot_shared_prefix_decode", "parrot_per_request_decode",
    "parrot_nested_prefix_decode", "parrot_shared_prefix_decode_append",
    "parrot_validate_inputs", "parrot_validate_nested_inputs",
    "parrot_prefill_workspace_bytes", "parrot_prefill_single_pass", "parrot_shared_prefix_prefill",
    "parrot_validate_prefill_inputs", "parrot_last_error", "parrot_abi_version",
    "parrot_shared_prefix_decode_noalloc", "parrot_hbm_read_ceiling", "parrot_mfma_issue_ceiling",
)

STATIC_SCRATCH_BYTES = 64 << 20   # PARROT_STATIC_SCRATCH_BYTES

_lib: Optional[ctypes.CDLL] = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the built library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2405_19888_amd.build` (no CPU fallback exists)")
    lib = ctypes.CDLL(path)
    vp, i32p, sz = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t
    prob_p = ctypes.POINTER(ParrotProblem)
    lib.parrot_workspace_bytes.argtypes = [prob_p]
    lib.parrot_workspace_bytes.restype = sz
    dec_args = [prob_p, vp, vp, vp, vp, vp, i32p, i32p, i32p, i32p, i32p, vp, vp, vp, sz, vp,
                ctypes.POINTER(ParrotTrace)]
    for name in ("parrot_shared_prefix_decode", "parrot_per_request_decode"):
        f = getattr(lib, name)
        f.argtypes = dec_args
        f.restype = ctypes.c_int
    lib.parrot_shared_prefix_decode_noalloc.argtypes = dec_args[:13] + dec_args[15:]
    lib.parrot_shared_prefix_decode_noalloc.restype = ctypes.c_int
    lib.parrot_shared_prefix_decode_append.argtypes = dec_args[:2] + [vp, vp] + dec_args[2:]
    lib.parrot_shared_prefix_decode_append.restype = ctypes.c_int
    lib.parrot_nested_prefix_decode.argtypes = dec_args[:8] + [i32p] + dec_args[8:]
    lib.parrot_nested_prefix_decode.restype = ctypes.c_int
    lib.parrot_validate_inputs.argtypes = [prob_p, i32p, i32p, i32p, i32p, i32p, vp, vp]
    lib.parrot_validate_inputs.restype = ctypes.c_int
    lib.parrot_validate_nested_inputs.argtypes = [prob_p, i32p, i32p, i32p, i32p, i32p, i32p,
                                                  vp, vp]
    lib.parrot_validate_nested_inputs.restype = ctypes.c_int
    rows_p = ctypes.POINTER(ParrotPrefillRows)
    lib.parrot_prefill_workspace_bytes.argtypes = [prob_p, rows_p]
    lib.parrot_prefill_workspace_bytes.restype = sz
    lib.parrot_shared_prefix_prefill.argtypes = [
        prob_p, rows_p, vp, i32p, vp, vp, vp, vp, i32p, i32p, i32p, i32p, i32p, i32p, vp, vp,
        vp, sz, vp, ctypes.POINTER(ParrotTrace)]
    lib.parrot_shared_prefix_prefill.restype = ctypes.c_int
    lib.parrot_validate_prefill_inputs.argtypes = [prob_p, rows_p, i32p, i32p, i32p, i32p,
                                                   i32p, i32p, i32p, vp, vp]
    lib.parrot_validate_prefill_inputs.restype = ctypes.c_int
    lib.parrot_prefill_single_pass.argtypes = [prob_p, rows_p, ctypes.c_int]
    lib.parrot_prefill_single_pass.restype = ctypes.c_int
    lib.parrot_hbm_read_ceiling.argtypes = [vp, sz, vp, ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_int32, vp, ctypes.POINTER(ParrotTrace)]
    lib.parrot_hbm_read_ceiling.restype = ctypes.c_int
    lib.parrot_mfma_issue_ceiling.argtypes = [vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, vp,
                                              ctypes.POINTER(ParrotTrace)]
    lib.parrot_mfma_issue_ceiling.restype = ctypes.c_int
    lib.parrot_last_error.argtypes = []
    lib.parrot_last_error.restype = ctypes.c_char_p
    lib.parrot_abi_version.argtypes = []
    lib.parrot_abi_version.restype = ctypes.c_int
    _lib = lib
    return lib


def parrot_last_error() -> str:
    return load_library().parrot_last_error().decode()


def parrot_abi_version() -> int:
    return load_library().parrot_abi_version()


def make_problem(*, num_requests, num_heads, head_dim, block_size, num_groups, max_group_size,
                 max_prefix_len, max_suffix_len, prefix_table_stride, suffix_table_stride,
                 num_prefix_blocks, num_suffix_blocks, dtype, sm_scale,
                 max_prefix_depth=0) -> ParrotProblem:
    code = DTYPE_CODES[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    return ParrotProblem(int(num_requests), int(num_heads), int(head_dim), int(block_size),
                         int(num_groups), int(max_group_size), int(max_prefix_len),
                         int(max_suffix_len), int(prefix_table_stride), int(suffix_table_stride),
                         int(num_prefix_blocks), int(num_suffix_blocks), code, float(sm_scale),
                         int(max_prefix_depth))


def parrot_workspace_bytes(problem: ParrotProblem) -> int:
    n = load_library().parrot_workspace_bytes(ctypes.byref(problem))
    if n == ctypes.c_size_t(-1).value:
        raise ParrotError(PARROT_ERR_INVALID_ARGUMENT, parrot_last_error())
    return int(n)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _check(status: int):
    if status != PARROT_OK:
        raise ParrotError(status, parrot_last_error())


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _decode(fn_name, problem, q, prefix_k, prefix_v, suffix_k, suffix_v, prefix_block_tables,
            prefix_lens, suffix_block_tables, suffix_lens, group_ids, out, lse, workspace,
            stream=None, trace: Optional[ParrotTrace] = None, prefix_parents=None):
    lib = load_library()
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    parents = (_ptr(prefix_parents),) if fn_name == "parrot_nested_prefix_decode" else ()
    status = getattr(lib, fn_name)(
        ctypes.byref(problem), _ptr(q), _ptr(prefix_k), _ptr(prefix_v), _ptr(suffix_k),
        _ptr(suffix_v), _ptr(prefix_block_tables), _ptr(prefix_lens), *parents,
        _ptr(suffix_block_tables), _ptr(suffix_lens), _ptr(group_ids), _ptr(out), _ptr(lse),
        _ptr(workspace), ws_bytes, _stream_handle(stream),
        ctypes.byref(trace) if trace is not None else None)
    _check(status)


def parrot_shared_prefix_decode(problem, q, prefix_k, prefix_v, suffix_k, suffix_v,
                                prefix_block_tables, prefix_lens, suffix_block_tables,
                                suffix_lens, group_ids, out, lse, workspace, stream=None,
                                trace=None):
    """Shared-prefix decode attention; writes ``out`` and ``lse`` (see the C header)."""
    _decode("parrot_shared_prefix_decode", problem, q, prefix_k, prefix_v, suffix_k, suffix_v,
            prefix_block_tables, prefix_lens, suffix_block_tables, suffix_lens, group_ids,
            out, lse, workspace, stream, trace)


def parrot_shared_prefix_decode_noalloc(problem, q, prefix_k, prefix_v, suffix_k, suffix_v,
                                        prefix_block_tables, prefix_lens, suffix_block_tables,
                                        suffix_lens, group_ids, out, lse, stream=None,
                                        trace=None):
    """Shared-prefix decode attention with the library's fixed partial-result
    array instead of a workspace (allocates nothing; see the C header)."""
    lib = load_library()
    _check(lib.parrot_shared_prefix_decode_noalloc(
        ctypes.byref(problem), _ptr(q), _ptr(prefix_k), _ptr(prefix_v), _ptr(suffix_k),
        _ptr(suffix_v), _ptr(prefix_block_tables), _ptr(prefix_lens), _ptr(suffix_block_tables),
        _ptr(suffix_lens), _ptr(group_ids), _ptr(out), _ptr(lse), _stream_handle(stream),
        ctypes.byref(trace) if trace is not None else None))


def parrot_mfma_issue_ceiling(sink, workgroups: int, iters: int, valu_x4: int = 0, stream=None,
                              trace=None):
    """Enqueue the matrix-core issue probe (8 x 16384 flop per wave and
    iteration, valu_x4 / 4 vector instructions per MFMA) folding into ``sink``."""
    _check(load_library().parrot_mfma_issue_ceiling(_ptr(sink), int(workgroups), int(iters),
                                                    int(valu_x4), _stream_handle(stream),
                                                    ctypes.byref(trace) if trace is not None else None))


def parrot_hbm_read_ceiling(src, sink, workgroups: int, loads_per_thread: int = 8,
                            wave_spans: bool = True, nbytes=None, stream=None, trace=None):
    """Enqueue the read-bandwidth probe over ``src`` (a device tensor; all of
    it unless ``nbytes``) folding into ``sink`` (a device uint32/int32);
    ``trace`` (a ParrotTrace) attaches its partials pair to the launch."""
    n = src.numel() * src.element_size() if nbytes is None else int(nbytes)
    _check(load_library().parrot_hbm_read_ceiling(_ptr(src), n, _ptr(sink), int(workgroups),
                                                  int(loads_per_thread), 1 if wave_spans else 0,
                                                  _stream_handle(stream),
                                                  ctypes.byref(trace) if trace is not None else None))


def parrot_per_request_decode(problem, q, prefix_k, prefix_v, suffix_k, suffix_v,
                              prefix_block_tables, prefix_lens, suffix_block_tables,
                              suffix_lens, group_ids, out, lse, workspace, stream=None,
                              trace=None):
    """Per-request (no sharing) decode attention over the same inputs."""
    _decode("parrot_per_request_decode", problem, q, prefix_k, prefix_v, suffix_k, suffix_v,
            prefix_block_tables, prefix_lens, suffix_block_tables, suffix_lens, group_ids,
            out, lse, workspace, stream, trace)


def parrot_shared_prefix_decode_append(problem, q, k_new, v_new, prefix_k, prefix_v, suffix_k,
                                       suffix_v, prefix_block_tables, prefix_lens,
                                       suffix_block_tables, suffix_lens, group_ids, out, lse,
                                       workspace, stream=None, trace=None):
    """Append this step's K/V (k_new, v_new) into the suffix pools, then
    shared-prefix decode attention (see the C header)."""
    lib = load_library()
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.parrot_shared_prefix_decode_append(
        ctypes.byref(problem), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(prefix_k), _ptr(prefix_v),
        _ptr(suffix_k), _ptr(suffix_v), _ptr(prefix_block_tables), _ptr(prefix_lens),
        _ptr(suffix_block_tables), _ptr(suffix_lens), _ptr(group_ids), _ptr(out), _ptr(lse),
        _ptr(workspace), ws_bytes, _stream_handle(stream),
        ctypes.byref(trace) if trace is not None else None))


def parrot_nested_prefix_decode(problem, q, prefix_k, prefix_v, suffix_k, suffix_v,
                                prefix_block_tables, prefix_lens, prefix_parents,
                                suffix_block_tables, suffix_lens, group_ids, out, lse, workspace,
                                stream=None, trace=None):
    """Shared-prefix decode attention with nested groups (see the C header)."""
    _decode("parrot_nested_prefix_decode", problem, q, prefix_k, prefix_v, suffix_k, suffix_v,
            prefix_block_tables, prefix_lens, suffix_block_tables, suffix_lens, group_ids,
            out, lse, workspace, stream, trace, prefix_parents=prefix_parents)


def parrot_validate_nested_inputs(problem, prefix_block_tables, prefix_lens, prefix_parents,
                                  suffix_block_tables, suffix_lens, group_ids, scratch,
                                  stream=None):
    """Device-side content check including the group parents (synchronises)."""
    lib = load_library()
    _check(lib.parrot_validate_nested_inputs(
        ctypes.byref(problem), _ptr(prefix_block_tables), _ptr(prefix_lens), _ptr(prefix_parents),
        _ptr(suffix_block_tables), _ptr(suffix_lens), _ptr(group_ids), _ptr(scratch),
        _stream_handle(stream)))


def parrot_validate_inputs(problem, prefix_block_tables, prefix_lens, suffix_block_tables,
                           suffix_lens, group_ids, scratch, stream=None):
    """Device-side content check (synchronises the stream)."""
    lib = load_library()
    _check(lib.parrot_validate_inputs(
        ctypes.byref(problem), _ptr(prefix_block_tables), _ptr(prefix_lens),
        _ptr(suffix_block_tables), _ptr(suffix_lens), _ptr(group_ids), _ptr(scratch),
        _stream_handle(stream)))


def make_prefill_rows(num_query_rows, max_query_rows, max_group_rows) -> ParrotPrefillRows:
    return ParrotPrefillRows(int(num_query_rows), int(max_query_rows), int(max_group_rows))


def prefill_rows_from_host(query_offsets, group_ids, num_groups, prefix_parents=None
                           ) -> ParrotPrefillRows:
    """Row counts of a prefill call from host copies of its offsets and groups."""
    import numpy as np
    off = np.asarray(query_offsets, dtype=np.int64)
    q = np.diff(off)
    per_group = np.zeros(max(int(num_groups), 1), dtype=np.int64)
    par = None if prefix_parents is None else np.asarray(prefix_parents)
    for r, g in enumerate(np.asarray(group_ids)):
        x = int(g)
        while x >= 0:
            per_group[x] += q[r]
            x = int(par[x]) if par is not None else -1
    return make_prefill_rows(int(off[-1]), max(int(q.max()) if q.size else 0, 1),
                             int(per_group.max()) if num_groups else 0)


def parrot_prefill_workspace_bytes(problem: ParrotProblem, rows: ParrotPrefillRows) -> int:
    n = load_library().parrot_prefill_workspace_bytes(ctypes.byref(problem), ctypes.byref(rows))
    if n == ctypes.c_size_t(-1).value:
        raise ParrotError(PARROT_ERR_INVALID_ARGUMENT, parrot_last_error())
    return int(n)


def parrot_prefill_single_pass(problem: ParrotProblem, rows: ParrotPrefillRows,
                               nested: bool = False) -> bool:
    """Whether the prefill entry point takes the single pass for these
    arguments (else partial results and the merge kernel)."""
    r = load_library().parrot_prefill_single_pass(ctypes.byref(problem), ctypes.byref(rows),
                                                  1 if nested else 0)
    if r < 0:
        raise ParrotError(PARROT_ERR_INVALID_ARGUMENT, parrot_last_error())
    return bool(r)


def parrot_shared_prefix_prefill(problem, rows, q, query_offsets, prefix_k, prefix_v, suffix_k,
                                 suffix_v, prefix_block_tables, prefix_lens, prefix_parents,
                                 suffix_block_tables, suffix_lens, group_ids, out, lse, workspace,
                                 stream=None, trace=None):
    """Prefill of forked contexts' new rows (see the C header); prefix_parents
    may be None for flat groups."""
    lib = load_library()
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.parrot_shared_prefix_prefill(
        ctypes.byref(problem), ctypes.byref(rows), _ptr(q), _ptr(query_offsets), _ptr(prefix_k),
        _ptr(prefix_v), _ptr(suffix_k), _ptr(suffix_v), _ptr(prefix_block_tables),
        _ptr(prefix_lens), _ptr(prefix_parents), _ptr(suffix_block_tables), _ptr(suffix_lens),
        _ptr(group_ids), _ptr(out), _ptr(lse), _ptr(workspace), ws_bytes, _stream_handle(stream),
        ctypes.byref(trace) if trace is not None else None))


def parrot_validate_prefill_inputs(problem, rows, query_offsets, prefix_block_tables, prefix_lens,
                                   prefix_parents, suffix_block_tables, suffix_lens, group_ids,
                                   scratch, stream=None):
    """Device-side content check of a prefill call's inputs (synchronises)."""
    lib = load_library()
    _check(lib.parrot_validate_prefill_inputs(
        ctypes.byref(problem), ctypes.byref(rows), _ptr(query_offsets), _ptr(prefix_block_tables),
        _ptr(prefix_lens), _ptr(prefix_parents), _ptr(suffix_block_tables), _ptr(suffix_lens),
        _ptr(group_ids), _ptr(scratch), _stream_handle(stream)))


def problem_from_host(*, num_heads, head_dim, block_size, dtype, sm_scale, group_ids, prefix_lens,
                      suffix_lens, prefix_table_stride, suffix_table_stride, num_prefix_blocks,
                      num_suffix_blocks, prefix_parents=None) -> ParrotProblem:
    """Fill a ParrotProblem from host copies of the batch metadata.

    ``group_ids``, ``prefix_lens``, ``suffix_lens`` (and, for nested groups,
    ``prefix_parents``) are host sequences; only their sizes, maxima and the
    group chains are used (the serving engine knows them on the host).
    """
    import numpy as np
    gid = np.asarray(group_ids)
    plen = np.asarray(prefix_lens)
    slen = np.asarray(suffix_lens)
    ng = int(plen.shape[0])
    readers = np.zeros(max(ng, 1), dtype=np.int64)
    depth = 1 if ng else 0
    par = None if prefix_parents is None else np.asarray(prefix_parents)
    # walks stop after ng steps: parents outside [-1, g) (which the validator
    # rejects) cannot loop them
    for g in gid:
        x, n = int(g), 0
        while 0 <= x < ng and n < ng:
            readers[x] += 1
            n += 1
            x = int(par[x]) if par is not None else -1
    # max_prefix_depth bounds every group's chain, read or not
    for g in range(ng if par is not None else 0):
        n, x = 0, g
        while 0 <= x < ng and n < ng:
            n += 1
            x = int(par[x])
        depth = max(depth, n)
    return make_problem(
        num_requests=gid.shape[0], num_heads=num_heads, head_dim=head_dim,
        block_size=block_size, num_groups=ng, max_group_size=int(readers.max()) if ng else 0,
        max_prefix_len=int(plen.max()) if ng else 0,
        max_suffix_len=int(slen.max()) if slen.size else 0,
        prefix_table_stride=prefix_table_stride, suffix_table_stride=suffix_table_stride,
        num_prefix_blocks=num_prefix_blocks, num_suffix_blocks=num_suffix_blocks,
        dtype=dtype, sm_scale=sm_scale, max_prefix_depth=depth if par is not None else 0)


class Decoder:
    """Owns the output, lse and workspace buffers for one problem shape."""

    def __init__(self, problem: ParrotProblem, device="cuda", out_dtype=None):
        self.problem = problem
        self.device = torch.device(device)
        inv = {v: k for k, v in DTYPE_CODES.items()}
        self.dtype = inv[problem.dtype] if out_dtype is None else out_dtype
        R, H, D = problem.num_requests, problem.num_heads, problem.head_dim
        self.out = torch.empty((R, H, D), dtype=self.dtype, device=self.device)
        self.lse = torch.empty((R, H), dtype=torch.float32, device=self.device)
        nbytes = parrot_workspace_bytes(problem)
        self.workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)

    @staticmethod
    def _entry(shared: bool, nested: bool, append: bool = False) -> str:
        if nested or append:
            if not shared or (nested and append):
                raise ValueError("nested groups and appending have shared-path entry points only")
            return "parrot_nested_prefix_decode" if nested else "parrot_shared_prefix_decode_append"
        return "parrot_shared_prefix_decode" if shared else "parrot_per_request_decode"

    def bind(self, t: dict, shared: bool = True, stream=None, nested: bool = False,
             append: bool = False):
        """Marshal the arguments once; the returned callable re-issues the same
        call (same tensors, stream and buffers) with only the optional trace.
        ``nested`` calls the nested-group entry point with t["prefix_parents"];
        ``append`` the appending one with t["k_new"], t["v_new"]."""
        lib = load_library()
        name = self._entry(shared, nested, append)
        fn = getattr(lib, name)
        pk = t.get("prefix_k", t.get("k_pool")); pv = t.get("prefix_v", t.get("v_pool"))
        sk = t.get("suffix_k", t.get("k_pool")); sv = t.get("suffix_v", t.get("v_pool"))
        ws = self.workspace
        parents = (_ptr(t["prefix_parents"]),) if nested else ()
        new_kv = (_ptr(t["k_new"]), _ptr(t["v_new"])) if append else ()
        args = (ctypes.byref(self.problem), _ptr(t["q"]), *new_kv, _ptr(pk), _ptr(pv), _ptr(sk),
                _ptr(sv), _ptr(t["prefix_tables"]), _ptr(t["prefix_lens"]), *parents,
                _ptr(t["suffix_tables"]), _ptr(t["suffix_lens"]), _ptr(t["group_ids"]),
                _ptr(self.out), _ptr(self.lse), _ptr(ws), ws.numel() * ws.element_size(),
                _stream_handle(stream))

        def call(trace: Optional[ParrotTrace] = None):
            _check(fn(*args, ctypes.byref(trace) if trace is not None else None))
        return call

    def __call__(self, t: dict, shared: bool = True, stream=None, trace=None, nested: bool = False,
                 append: bool = False):
        if append:
            self.bind(t, shared=shared, stream=stream, append=True)(trace)
            return self.out, self.lse
        _decode(self._entry(shared, nested), self.problem, t["q"],
                t.get("prefix_k", t.get("k_pool")), t.get("prefix_v", t.get("v_pool")),
                t.get("suffix_k", t.get("k_pool")), t.get("suffix_v", t.get("v_pool")),
                t["prefix_tables"], t["prefix_lens"], t["suffix_tables"], t["suffix_lens"],
                t["group_ids"], self.out, self.lse, self.workspace, stream=stream, trace=trace,
                prefix_parents=t.get("prefix_parents") if nested else None)
        return self.out, self.lse


class Prefiller:
    """Owns the output, lse and workspace buffers of one prefill shape."""

    def __init__(self, problem: ParrotProblem, rows: ParrotPrefillRows, device="cuda"):
        self.problem = problem
        self.rows = rows
        self.device = torch.device(device)
        inv = {v: k for k, v in DTYPE_CODES.items()}
        self.dtype = inv[problem.dtype]
        T, H, D = rows.num_query_rows, problem.num_heads, problem.head_dim
        self.out = torch.empty((T, H, D), dtype=self.dtype, device=self.device)
        self.lse = torch.empty((T, H), dtype=torch.float32, device=self.device)
        nbytes = parrot_prefill_workspace_bytes(problem, rows)
        self.workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)

    def bind(self, t: dict, stream=None, nested: bool = False):
        """Marshal once; the returned callable re-issues the same call.  ``t``
        holds q_rows, query_offsets, the pools (k_pool / v_pool or
        prefix_k ... suffix_v) and the int arrays; ``nested`` passes
        t["prefix_parents"]."""
        fn = load_library().parrot_shared_prefix_prefill
        ws = self.workspace
        args = (ctypes.byref(self.problem), ctypes.byref(self.rows), _ptr(t["q_rows"]),
                _ptr(t["query_offsets"]), _ptr(t.get("prefix_k", t.get("k_pool"))),
                _ptr(t.get("prefix_v", t.get("v_pool"))), _ptr(t.get("suffix_k", t.get("k_pool"))),
                _ptr(t.get("suffix_v", t.get("v_pool"))), _ptr(t["prefix_tables"]),
                _ptr(t["prefix_lens"]), _ptr(t["prefix_parents"]) if nested else None,
                _ptr(t["suffix_tables"]), _ptr(t["suffix_lens"]), _ptr(t["group_ids"]),
                _ptr(self.out), _ptr(self.lse), _ptr(ws), ws.numel() * ws.element_size(),
                _stream_handle(stream))

        def call(trace: Optional[ParrotTrace] = None):
            _check(fn(*args, ctypes.byref(trace) if trace is not None else None))
        return call

    def __call__(self, t: dict, stream=None, trace=None, nested: bool = False):
        self.bind(t, stream=stream, nested=nested)(trace)
        return self.out, self.lse


def _sizes_from_tensors(q, prefix_k, suffix_k, prefix_tables, suffix_tables, group_ids,
                        prefix_lens, suffix_lens, sm_scale, prefix_parents):
    """ParrotProblem of a call given as torch tensors (one device-to-host copy
    of the group ids and lengths, for the maxima and group sizes)."""
    return problem_from_host(
        num_heads=q.shape[-2], head_dim=q.shape[-1], block_size=suffix_k.shape[2],
        dtype=q.dtype, sm_scale=sm_scale, group_ids=group_ids.cpu().numpy(),
        prefix_lens=prefix_lens.cpu().numpy(), suffix_lens=suffix_lens.cpu().numpy(),
        prefix_table_stride=prefix_tables.shape[1] if prefix_tables.dim() == 2 else 0,
        suffix_table_stride=suffix_tables.shape[1],
        num_prefix_blocks=prefix_k.shape[0], num_suffix_blocks=suffix_k.shape[0],
        prefix_parents=None if prefix_parents is None else prefix_parents.cpu().numpy())


def shared_prefix_decode(q, prefix_k, prefix_v, suffix_k, suffix_v, prefix_tables, prefix_lens,
                         suffix_tables, suffix_lens, group_ids, *, sm_scale, prefix_parents=None,
                         per_request=False, stream=None):
    """One decode call on torch tensors laid out as the C entry points take
    them (q [R, H, D]; pools [blocks, H, 16, D]; int32 tables, lengths, group
    ids and, for nested groups, parents).  Sizes the problem from host copies
    of the group ids and lengths, allocates out, lse and the workspace, and
    runs on ``stream`` (default: the current stream).  Returns (out, lse).
    ``per_request`` runs the baseline that reads each request's prefix itself.
    Engines that know the maxima on the host should build a ParrotProblem and
    reuse a Decoder instead (no copy, no allocation per call)."""
    prob = _sizes_from_tensors(q, prefix_k, suffix_k, prefix_tables, suffix_tables, group_ids,
                               prefix_lens, suffix_lens, sm_scale, prefix_parents)
    dec = Decoder(prob, device=q.device)
    t = dict(q=q, prefix_k=prefix_k, prefix_v=prefix_v, suffix_k=suffix_k, suffix_v=suffix_v,
             prefix_tables=prefix_tables, prefix_lens=prefix_lens, suffix_tables=suffix_tables,
             suffix_lens=suffix_lens, group_ids=group_ids, prefix_parents=prefix_parents)
    return dec(t, shared=not per_request, stream=stream, nested=prefix_parents is not None)


def shared_prefix_prefill(q_rows, query_offsets, prefix_k, prefix_v, suffix_k, suffix_v,
                          prefix_tables, prefix_lens, suffix_tables, suffix_lens, group_ids, *,
                          sm_scale, prefix_parents=None, stream=None):
    """One prefill call on torch tensors: rows [query_offsets[r],
    query_offsets[r+1]) of q_rows [T, H, D] are request r's last own tokens.
    Sizes the problem and the row counts from host copies of the int arrays,
    allocates out, lse and the workspace, and runs on ``stream``.  Returns
    (out, lse)."""
    prob = _sizes_from_tensors(q_rows, prefix_k, suffix_k, prefix_tables, suffix_tables, group_ids,
                               prefix_lens, suffix_lens, sm_scale, prefix_parents)
    rows = prefill_rows_from_host(query_offsets.cpu().numpy(), group_ids.cpu().numpy(),
                                  prob.num_groups,
                                  None if prefix_parents is None else prefix_parents.cpu().numpy())
    pre = Prefiller(prob, rows, device=q_rows.device)
    t = dict(q_rows=q_rows, query_offsets=query_offsets, prefix_k=prefix_k, prefix_v=prefix_v,
             suffix_k=suffix_k, suffix_v=suffix_v, prefix_tables=prefix_tables,
             prefix_lens=prefix_lens, suffix_tables=suffix_tables, suffix_lens=suffix_lens,
             group_ids=group_ids, prefix_parents=prefix_parents)
    return pre(t, stream=stream, nested=prefix_parents is not None)
