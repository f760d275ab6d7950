"""The C ABI on the host: the library loads, exports every declared symbol,
sizes workspaces, and rejects bad arguments before any device work.
Runs without a GPU (no call here reaches a kernel launch)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2405_19888_amd import binding as B

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")


def declared_functions():
    names = set()
    for h in sorted(os.listdir(INCLUDE)):
        if h.endswith(".h"):
            text = open(os.path.join(INCLUDE, h)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(parrot_\w+)\s*\(", text))
    return sorted(names)


def test_exports_every_declared_symbol(parrot_lib):
    from paper_2405_19888_amd.context import STORE_EXPORTED
    names = declared_functions()
    assert set(names) == set(B.EXPORTED) | set(STORE_EXPORTED), names
    for n in names:
        assert hasattr(parrot_lib, n), f"{n} not exported"


def declared_arities():
    """Parameter count of every function declared in include/*.h."""
    out = {}
    for h in sorted(os.listdir(INCLUDE)):
        if not h.endswith(".h"):
            continue
        text = open(os.path.join(INCLUDE, h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for m in re.finditer(r"\b(parrot_\w+)\s*\(([^;{]*?)\)\s*;", text):
            params = " ".join(m.group(2).split())
            out[m.group(1)] = 0 if params in ("", "void") else params.count(",") + 1
    return out


def test_binding_matches_header_arity(parrot_lib):
    """Every function of the C header is bound with as many arguments as it
    declares (argument lists drift silently through ctypes otherwise)."""
    from paper_2405_19888_amd import context
    context._lib()                       # binds the context-store functions
    arity = declared_arities()
    assert set(arity) == set(declared_functions()), "declarations the parser missed"
    for name, n in arity.items():
        f = getattr(parrot_lib, name)
        assert f.argtypes is not None, f"{name} has no argtypes"
        assert len(f.argtypes) == n, f"{name}: header {n} arguments, binding {len(f.argtypes)}"


def test_abi_version(parrot_lib):
    assert B.parrot_abi_version() == 8


def test_batches_above_1024_requests_are_sized(parrot_lib):
    """No per-call request cap: decode and prefill size batches of any count
    (the split-KV role streams them in slices of 1024 requests)."""
    for R in (1024, 1025, 2500, 20000):
        w = B.parrot_workspace_bytes(base_problem(num_requests=R))
        assert w >= R * 32 * 129 * 4, R
        rows = B.make_prefill_rows(R, 1, R)
        assert B.parrot_prefill_workspace_bytes(base_problem(num_requests=R), rows) > 0


def test_read_ceiling_rejects_bad_arguments_without_a_device(parrot_lib):
    f = parrot_lib.parrot_hbm_read_ceiling
    buf = ctypes.create_string_buffer(64)
    base = ctypes.addressof(buf) + (-ctypes.addressof(buf)) % 16
    assert f(None, 16, base, 1, 8, 1, None, None) == B.PARROT_ERR_INVALID_ARGUMENT
    assert f(base, 16, None, 1, 8, 1, None, None) == B.PARROT_ERR_INVALID_ARGUMENT
    assert f(base + 8, 16, base, 1, 8, 1, None, None) == B.PARROT_ERR_INVALID_ARGUMENT     # misaligned
    assert f(base, 20, base, 1, 8, 1, None, None) == B.PARROT_ERR_INVALID_ARGUMENT         # not 16 x n
    assert f(base, 16, base, 0, 8, 1, None, None) == B.PARROT_ERR_INVALID_ARGUMENT         # no workgroups
    assert f(base, 16, base, 1, 8, 2, None, None) == B.PARROT_ERR_INVALID_ARGUMENT         # order flag
    assert f(base, 16, base, 1, 5, 1, None, None) == B.PARROT_ERR_UNSUPPORTED
    assert "loads_per_thread" in B.parrot_last_error()


def test_mfma_issue_ceiling_rejects_bad_arguments_without_a_device(parrot_lib):
    f = parrot_lib.parrot_mfma_issue_ceiling
    buf = ctypes.create_string_buffer(16)
    base = ctypes.addressof(buf) + (-ctypes.addressof(buf)) % 4
    assert f(None, 1, 1, 0, None, None) == B.PARROT_ERR_INVALID_ARGUMENT
    assert f(base + 2, 1, 1, 0, None, None) == B.PARROT_ERR_INVALID_ARGUMENT     # misaligned
    assert f(base, 0, 1, 0, None, None) == B.PARROT_ERR_INVALID_ARGUMENT         # no workgroups
    assert f(base, 1, 0, 0, None, None) == B.PARROT_ERR_INVALID_ARGUMENT         # no iterations
    assert f(base, 1, 1, 9, None, None) == B.PARROT_ERR_UNSUPPORTED
    assert "valu_x4" in B.parrot_last_error()


def test_noalloc_refuses_batches_above_its_array_without_a_device(parrot_lib):
    """The allocation-free entry point sizes the call on the host and refuses
    one whose partial results exceed the library's fixed array before it
    touches the device (pointers are never read)."""
    big = base_problem(num_requests=512, num_groups=8, max_group_size=64, max_prefix_len=4096,
                       prefix_table_stride=256, max_suffix_len=4096, suffix_table_stride=256)
    st = parrot_lib.parrot_shared_prefix_decode_noalloc(
        ctypes.byref(big), *([None] * 12), None, None)
    assert st == B.PARROT_ERR_WORKSPACE_TOO_SMALL
    assert "fixed array" in B.parrot_last_error()
    st = parrot_lib.parrot_shared_prefix_decode_noalloc(
        ctypes.byref(base_problem(num_requests=0)), *([None] * 12), None, None)
    assert st == B.PARROT_OK
    st = parrot_lib.parrot_shared_prefix_decode_noalloc(None, *([None] * 12), None, None)
    assert st == B.PARROT_ERR_INVALID_ARGUMENT


def base_problem(**over):
    kw = dict(num_requests=32, num_heads=32, head_dim=128, block_size=16, num_groups=1,
              max_group_size=32, max_prefix_len=2048, max_suffix_len=512,
              prefix_table_stride=128, suffix_table_stride=32, num_prefix_blocks=1000,
              num_suffix_blocks=1000, dtype=1, sm_scale=0.088)
    kw.update(over)
    return B.make_problem(**kw)


def test_struct_layout_matches_header():
    assert ctypes.sizeof(B.ParrotProblem) == 15 * 4
    assert ctypes.sizeof(B.ParrotTrace) == 4 * ctypes.sizeof(ctypes.c_void_p)
    assert ctypes.sizeof(B.ParrotPrefillRows) == 3 * 4


def test_workspace_sizes(parrot_lib):
    assert B.parrot_workspace_bytes(base_problem(num_requests=0)) == 0
    w0 = B.parrot_workspace_bytes(base_problem())
    # 2048/256 prefix slots + 512/128 suffix slots, each D + 1 floats
    assert w0 >= 32 * 32 * (8 + 4) * 129 * 4
    # (not num_heads: the split-KV grid is fixed per device, so more heads
    # means fewer column groups per head, and at most that many pieces each)
    for field, bigger in [("num_requests", 64), ("max_prefix_len", 4096),
                          ("max_suffix_len", 1024), ("head_dim", 128)]:
        kw = {field: bigger}
        if field == "max_prefix_len":
            kw["prefix_table_stride"] = 256
        if field == "max_suffix_len":
            kw["suffix_table_stride"] = 64
        assert B.parrot_workspace_bytes(base_problem(**kw)) >= w0, field
    assert B.parrot_workspace_bytes(base_problem(head_dim=64)) < w0


@pytest.mark.parametrize("base", [
    dict(num_requests=4, num_heads=4, head_dim=64, dtype=0, max_group_size=4, max_prefix_len=128,
         prefix_table_stride=8, max_suffix_len=32, suffix_table_stride=2),     # tiny: small chunks
    dict(num_requests=4, num_heads=1, head_dim=64, dtype=0, max_group_size=4, max_prefix_len=1024,
         prefix_table_stride=64, max_suffix_len=32, suffix_table_stride=2),     # many small chunks
    dict(),                                                                      # LLaMA-7B, 1 x 32
])
def test_workspace_monotone_in_batch(parrot_lib, base):
    """A workspace sized for the largest batch serves every smaller one: the
    size never drops as requests or own tokens are added (the prefix chunk,
    which can grow with the own-token stream, does not shrink the slots)."""
    prev = 0
    g = base.get("max_group_size", 32)                   # requests >= the largest group
    for R in (g, g + 1, g + 3, 2 * g, 4 * g, 8 * g, 16 * g):
        w = B.parrot_workspace_bytes(base_problem(**dict(base, num_requests=R)))
        assert w >= prev, R
        prev = w
    prev = 0
    for S in (1, 2, 16, 32, 64, 100, 256, 512, 1024, 4096, 8192, 16384):
        w = B.parrot_workspace_bytes(base_problem(**dict(base, max_suffix_len=S,
                                                         suffix_table_stride=-(-S // 16))))
        assert w >= prev, S
        prev = w


@pytest.mark.parametrize("over,status,msg", [
    (dict(head_dim=96), B.PARROT_ERR_UNSUPPORTED, "head_dim"),
    (dict(block_size=32), B.PARROT_ERR_UNSUPPORTED, "block_size"),
    (dict(dtype=7), B.PARROT_ERR_UNSUPPORTED, "dtype"),
    (dict(num_heads=0), B.PARROT_ERR_INVALID_ARGUMENT, "num_heads"),
    (dict(num_requests=-1), B.PARROT_ERR_INVALID_ARGUMENT, "num_requests"),
    (dict(prefix_table_stride=10), B.PARROT_ERR_INVALID_ARGUMENT, "prefix_table_stride"),
    (dict(suffix_table_stride=1), B.PARROT_ERR_INVALID_ARGUMENT, "suffix_table_stride"),
    (dict(max_group_size=0), B.PARROT_ERR_INVALID_ARGUMENT, "max_group_size"),
    (dict(max_group_size=33), B.PARROT_ERR_INVALID_ARGUMENT, "max_group_size"),
    (dict(sm_scale=float("nan")), B.PARROT_ERR_INVALID_ARGUMENT, "sm_scale"),
    (dict(num_groups=0, max_suffix_len=0, suffix_table_stride=0), B.PARROT_ERR_INVALID_ARGUMENT,
     "non-empty"),
    (dict(max_prefix_depth=5), B.PARROT_ERR_UNSUPPORTED, "max_prefix_depth"),
    (dict(max_prefix_depth=-1), B.PARROT_ERR_INVALID_ARGUMENT, "max_prefix_depth"),
])
def test_bad_problem_rejected(parrot_lib, over, status, msg):
    with pytest.raises(B.ParrotError) as e:
        B.parrot_workspace_bytes(base_problem(**over))
    assert msg in str(e.value)
    # the decode entry points report the same status before touching the device
    st = parrot_lib.parrot_shared_prefix_decode(ctypes.byref(base_problem(**over)), *([None] * 13),
                                                0, None, None)
    assert st == status and msg in B.parrot_last_error()


FAKE = 1 << 20          # aligned fake device addresses: never dereferenced here


def call(lib, prob, fn="parrot_shared_prefix_decode", **ptrs):
    names = ["q", "pk", "pv", "sk", "sv", "ptab", "plen", "stab", "slen", "gid", "out", "lse", "ws"]
    if fn == "parrot_nested_prefix_decode":
        names.insert(7, "parents")
    if fn == "parrot_shared_prefix_decode_append":
        names[1:1] = ["k_new", "v_new"]
    vals = {n: FAKE + 4096 * i for i, n in enumerate(names)}
    vals.update(ptrs)
    ws_bytes = ptrs.get("ws_bytes", 1 << 40)
    vals.pop("ws_bytes", None)
    return getattr(lib, fn)(ctypes.byref(prob), *[vals[n] for n in names], ws_bytes, None, None)


_COMMON_FIELDS = ["q", "sk", "sv", "stab", "slen", "gid", "out", "lse", "ws", "pk", "pv", "ptab",
                  "plen"]
_NULL_CASES = [(fn, f) for fn in ("parrot_shared_prefix_decode", "parrot_per_request_decode",
                                  "parrot_nested_prefix_decode",
                                  "parrot_shared_prefix_decode_append")
               for f in _COMMON_FIELDS] + \
    [("parrot_nested_prefix_decode", "parents"), ("parrot_shared_prefix_decode_append", "k_new"),
     ("parrot_shared_prefix_decode_append", "v_new")]


@pytest.mark.parametrize("fn,field", _NULL_CASES)
def test_null_pointer_rejected(parrot_lib, fn, field):
    """Every pointer argument an entry point takes (prefix_parents only the
    nested one, k_new / v_new only the appending one) is checked for NULL."""
    st = call(parrot_lib, base_problem(max_prefix_depth=2), fn, **{field: None})
    assert st == B.PARROT_ERR_INVALID_ARGUMENT
    assert "NULL" in B.parrot_last_error()


@pytest.mark.parametrize("field,off", [("q", 8), ("out", 2), ("sk", 4), ("ws", 128), ("lse", 2),
                                       ("gid", 1)])
def test_misaligned_pointer_rejected(parrot_lib, field, off):
    st = call(parrot_lib, base_problem(), **{field: FAKE + off})
    assert st == B.PARROT_ERR_INVALID_ARGUMENT
    assert "aligned" in B.parrot_last_error()


def test_nested_workspace_grows_with_depth(parrot_lib):
    w1 = B.parrot_workspace_bytes(base_problem())
    assert B.parrot_workspace_bytes(base_problem(max_prefix_depth=1)) == w1
    w2 = B.parrot_workspace_bytes(base_problem(max_prefix_depth=2))
    w4 = B.parrot_workspace_bytes(base_problem(max_prefix_depth=4))
    # one slot stride serves both paths: the per-request path's pieces often
    # dominate, so deeper nesting never shrinks the workspace
    assert w1 <= w2 <= w4


def test_nested_entry_checks_like_the_flat_one(parrot_lib):
    prob = base_problem(max_prefix_depth=2)
    need = B.parrot_workspace_bytes(prob)
    st = call(parrot_lib, prob, "parrot_nested_prefix_decode", ws_bytes=need - 1)
    assert st == B.PARROT_ERR_WORKSPACE_TOO_SMALL
    st = call(parrot_lib, prob, "parrot_nested_prefix_decode", parents=FAKE + 2)
    assert st == B.PARROT_ERR_INVALID_ARGUMENT and "aligned" in B.parrot_last_error()


def test_append_inputs_must_be_aligned(parrot_lib):
    st = call(parrot_lib, base_problem(), "parrot_shared_prefix_decode_append", k_new=FAKE + 8)
    assert st == B.PARROT_ERR_INVALID_ARGUMENT and "k_new" in B.parrot_last_error()


def test_workspace_too_small(parrot_lib):
    prob = base_problem()
    need = B.parrot_workspace_bytes(prob)
    st = call(parrot_lib, prob, ws_bytes=need - 1)
    assert st == B.PARROT_ERR_WORKSPACE_TOO_SMALL
    assert str(need) in B.parrot_last_error()


def test_prefix_pointers_optional_without_groups(parrot_lib):
    prob = base_problem(num_groups=0, max_group_size=0, max_prefix_len=0, num_requests=0)
    assert call(parrot_lib, prob, pk=None, pv=None, ptab=None, plen=None) == B.PARROT_OK


def test_empty_batch_is_ok_without_device(parrot_lib):
    prob = base_problem(num_requests=0)
    assert call(parrot_lib, prob, q=None, out=None, lse=None, ws=None, ws_bytes=0) == B.PARROT_OK
    assert B.parrot_last_error() == ""


def test_missing_library_fails_loudly(tmp_path):
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        B._lib_saved = B._lib
        try:
            B._lib = None
            B.load_library(str(tmp_path / "nope.so"))
        finally:
            B._lib = B._lib_saved


# ------------------------------------------------------------------ prefill
def prefill_rows(**over):
    kw = dict(num_query_rows=32 * 256, max_query_rows=256, max_group_rows=32 * 256)
    kw.update(over)
    return B.make_prefill_rows(**kw)


def prefill_call(lib, prob, rows, **ptrs):
    names = ["q", "qoff", "pk", "pv", "sk", "sv", "ptab", "plen", "parents", "stab", "slen",
             "gid", "out", "lse", "ws"]
    vals = {n: FAKE + 4096 * i for i, n in enumerate(names)}
    vals.update(ptrs)
    ws_bytes = ptrs.get("ws_bytes", 1 << 40)
    vals.pop("ws_bytes", None)
    return lib.parrot_shared_prefix_prefill(ctypes.byref(prob), ctypes.byref(rows),
                                            *[vals[n] for n in names], ws_bytes, None, None)


def test_prefill_workspace_sizes(parrot_lib):
    prob = base_problem()
    assert B.parrot_prefill_workspace_bytes(prob, prefill_rows(num_query_rows=0)) == 0
    w = B.parrot_prefill_workspace_bytes(prob, prefill_rows())
    # at least one prefix slot and one own slot per (row, head), D + 1 floats
    # each, plus a 16-byte descriptor per row
    T, H, D = 32 * 256, 32, 128
    assert w >= T * H * 2 * (D + 1) * 4 + T * 16
    assert B.parrot_prefill_workspace_bytes(prob, prefill_rows(num_query_rows=32 * 128,
                                                               max_query_rows=128,
                                                               max_group_rows=32 * 128)) < w
    # nested groups need a slot range per level
    assert B.parrot_prefill_workspace_bytes(base_problem(max_prefix_depth=3), prefill_rows()) > w


def test_prefill_single_pass_choice(parrot_lib, monkeypatch):
    """The single pass needs flat groups, 16-bit caches and lengths within one
    8192-token chunk; by default it also needs tiles enough to fill the device
    without cutting the ranges into chunks (256 CUs assumed without a GPU)."""
    monkeypatch.delenv("PARROT_PREFILL_SINGLE_PASS", raising=False)
    prob, rows = base_problem(), prefill_rows()
    assert B.parrot_prefill_single_pass(prob, rows)                   # 64 row tiles x 32 heads
    assert not B.parrot_prefill_single_pass(prob, rows, nested=True)
    assert not B.parrot_prefill_single_pass(base_problem(dtype=0), rows)
    assert B.parrot_prefill_single_pass(base_problem(dtype=2), rows)
    few = prefill_rows(num_query_rows=32 * 16, max_query_rows=16, max_group_rows=32 * 16)
    assert not B.parrot_prefill_single_pass(prob, few)                # 4 tiles: chunked
    long_prefix = base_problem(max_prefix_len=9000, prefix_table_stride=563)
    assert not B.parrot_prefill_single_pass(long_prefix, rows)        # two 8192-token chunks
    monkeypatch.setenv("PARROT_PREFILL_SINGLE_PASS", "1")
    assert B.parrot_prefill_single_pass(prob, few)
    assert not B.parrot_prefill_single_pass(long_prefix, rows)
    assert not B.parrot_prefill_single_pass(prob, rows, nested=True)
    assert not B.parrot_prefill_single_pass(base_problem(dtype=0), few)
    monkeypatch.setenv("PARROT_PREFILL_SINGLE_PASS", "yes")                # not 0 or 1: the plan decides
    assert not B.parrot_prefill_single_pass(prob, few)
    monkeypatch.setenv("PARROT_PREFILL_SINGLE_PASS", "0")
    assert not B.parrot_prefill_single_pass(prob, rows)
    # the workspace bound does not depend on the plan
    w = B.parrot_prefill_workspace_bytes(prob, rows)
    monkeypatch.setenv("PARROT_PREFILL_SINGLE_PASS", "1")
    assert B.parrot_prefill_workspace_bytes(prob, rows) == w
    with pytest.raises(B.ParrotError, match="max_query_rows"):
        B.parrot_prefill_single_pass(prob, prefill_rows(max_query_rows=0))


@pytest.mark.parametrize("over,msg", [
    (dict(num_query_rows=-1), "num_query_rows"),
    (dict(max_query_rows=0), "max_query_rows"),
    (dict(max_query_rows=513), "max_query_rows"),
    (dict(num_query_rows=32 * 256 + 1, max_group_rows=0), "num_query_rows"),
    (dict(max_group_rows=32 * 256 + 1), "max_group_rows"),
    (dict(max_group_rows=-1), "max_group_rows"),
])
def test_prefill_bad_rows_rejected(parrot_lib, over, msg):
    with pytest.raises(B.ParrotError) as e:
        B.parrot_prefill_workspace_bytes(base_problem(), prefill_rows(**over))
    assert msg in str(e.value)
    st = prefill_call(parrot_lib, base_problem(), prefill_rows(**over))
    assert st == B.PARROT_ERR_INVALID_ARGUMENT and msg in B.parrot_last_error()


def test_prefill_ignores_max_group_size(parrot_lib):
    """Prefill bounds group rows through max_group_rows instead."""
    w = B.parrot_prefill_workspace_bytes(base_problem(max_group_size=0), prefill_rows())
    assert w == B.parrot_prefill_workspace_bytes(base_problem(), prefill_rows())


@pytest.mark.parametrize("field", ["q", "qoff", "sk", "sv", "stab", "slen", "gid", "out", "lse",
                                   "ws", "pk", "pv", "ptab", "plen"])
def test_prefill_null_pointer_rejected(parrot_lib, field):
    st = prefill_call(parrot_lib, base_problem(), prefill_rows(), **{field: None})
    assert st == B.PARROT_ERR_INVALID_ARGUMENT and "NULL" in B.parrot_last_error()


def test_prefill_parents_optional_but_aligned(parrot_lib):
    prob, rows = base_problem(), prefill_rows()
    need = B.parrot_prefill_workspace_bytes(prob, rows)
    assert prefill_call(parrot_lib, prob, rows, parents=FAKE + 2) == B.PARROT_ERR_INVALID_ARGUMENT
    assert "aligned" in B.parrot_last_error()
    st = prefill_call(parrot_lib, prob, rows, parents=None, ws_bytes=need - 1)
    assert st == B.PARROT_ERR_WORKSPACE_TOO_SMALL and str(need) in B.parrot_last_error()


def test_prefill_no_rows_is_ok_without_device(parrot_lib):
    st = prefill_call(parrot_lib, base_problem(), prefill_rows(num_query_rows=0), q=None,
                      out=None, lse=None, ws=None, ws_bytes=0)
    assert st == B.PARROT_OK and B.parrot_last_error() == ""


def test_prefill_rows_from_host():
    off = [0, 3, 3, 10, 12]
    rows = B.prefill_rows_from_host(off, group_ids=[0, 1, 1, -1], num_groups=2,
                                    prefix_parents=[-1, 0])
    assert (rows.num_query_rows, rows.max_query_rows, rows.max_group_rows) == (12, 7, 10)
    flat = B.prefill_rows_from_host(off, group_ids=[0, 1, 1, -1], num_groups=2)
    assert flat.max_group_rows == 7


def test_problem_from_host_sizes_every_chain():
    """max_prefix_depth covers every group's chain, also one that no request
    reads; max_group_size counts each group's members and descendants'."""
    common = dict(num_heads=2, head_dim=128, block_size=16, dtype=1, sm_scale=0.1,
                  prefix_table_stride=8, suffix_table_stride=8, num_prefix_blocks=64,
                  num_suffix_blocks=64)
    # groups 0 <- 1 <- 2 <- 3; requests read only groups 0 and 1
    p = B.problem_from_host(group_ids=[0, 1, 1, -1], prefix_lens=[16, 16, 16, 16],
                            suffix_lens=[1, 2, 3, 4], prefix_parents=[-1, 0, 1, 2], **common)
    assert p.max_prefix_depth == 4
    assert p.max_group_size == 3          # group 0: its member and group 1's two
    flat = B.problem_from_host(group_ids=[0, 1, 1, -1], prefix_lens=[16, 16, 16, 16],
                               suffix_lens=[1, 2, 3, 4], **common)
    assert (flat.max_prefix_depth, flat.max_group_size) == (0, 2)
    # a parent outside [-1, g) (rejected later by the validator) must not hang
    cyc = B.problem_from_host(group_ids=[0], prefix_lens=[16, 16], suffix_lens=[1],
                              prefix_parents=[1, 0], **common)
    assert cyc.max_prefix_depth <= 2
