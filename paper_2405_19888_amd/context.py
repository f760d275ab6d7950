"""ctypes binding of the host-side context store (include/parrot_context.h).

The store decides which prompt prefixes are shared (a trie of prefixes split
where semantic variables end), owns the paged KV block ids, and emits the
arrays the nested decode entry point takes.  Argument marshalling only.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Sequence

import numpy as np

from .binding import ParrotError, _check, load_library

STORE_EXPORTED = (
    "parrot_store_create", "parrot_store_destroy", "parrot_store_fill", "parrot_store_append",
    "parrot_store_free", "parrot_store_free_blocks", "parrot_store_num_prefixes",
    "parrot_store_prefix_tokens", "parrot_store_own_tokens", "parrot_store_batch_shape",
    "parrot_store_build_batch",
)


class BatchShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "num_groups", "max_group_size", "max_prefix_len", "max_suffix_len", "max_prefix_depth",
        "prefix_table_stride", "suffix_table_stride")]


def _lib():
    lib = load_library()
    if getattr(lib, "_store_bound", False):
        return lib
    i32, vp, p = ctypes.c_int32, ctypes.c_void_p, ctypes.POINTER
    ip = p(ctypes.c_int32)
    lib.parrot_store_create.argtypes = [i32, i32]
    lib.parrot_store_create.restype = vp
    lib.parrot_store_destroy.argtypes = [vp]
    lib.parrot_store_destroy.restype = None
    lib.parrot_store_fill.argtypes = [vp, ip, i32, ip, i32]
    lib.parrot_store_fill.restype = i32
    lib.parrot_store_append.argtypes = [vp, i32, i32]
    lib.parrot_store_append.restype = ctypes.c_int
    lib.parrot_store_free.argtypes = [vp, i32]
    lib.parrot_store_free.restype = ctypes.c_int
    for name in ("parrot_store_free_blocks", "parrot_store_num_prefixes"):
        getattr(lib, name).argtypes = [vp]
        getattr(lib, name).restype = i32
    for name in ("parrot_store_prefix_tokens", "parrot_store_own_tokens"):
        getattr(lib, name).argtypes = [vp, i32]
        getattr(lib, name).restype = i32
    lib.parrot_store_batch_shape.argtypes = [vp, ip, i32, p(BatchShape)]
    lib.parrot_store_batch_shape.restype = ctypes.c_int
    lib.parrot_store_build_batch.argtypes = [vp, ip, i32, i32, ip, ip, ip, ip, ip, ip]
    lib.parrot_store_build_batch.restype = ctypes.c_int
    lib._store_bound = True
    return lib


def _ints(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _iptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


@dataclass
class Batch:
    """Host arrays of one decode batch (see parrot_store_build_batch)."""
    group_ids: np.ndarray
    suffix_lens: np.ndarray
    suffix_tables: np.ndarray
    prefix_lens: np.ndarray
    prefix_parents: np.ndarray
    prefix_tables: np.ndarray
    shape: BatchShape


class ContextStore:
    """Prefix trie + KV block allocator over `num_blocks` blocks of `block_size`."""

    def __init__(self, block_size: int, num_blocks: int):
        self._lib = _lib()
        self._h = self._lib.parrot_store_create(int(block_size), int(num_blocks))
        if not self._h:
            raise ValueError("bad store arguments")
        self.block_size = int(block_size)
        self.num_blocks = int(num_blocks)

    def close(self):
        if self._h:
            self._lib.parrot_store_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def fill(self, tokens: Sequence[int], boundaries: Sequence[int] = ()) -> int:
        """Register a prompt; returns its context id.  Raises MemoryError when
        the free blocks do not suffice."""
        t, b = _ints(tokens), _ints(boundaries)
        c = self._lib.parrot_store_fill(self._h, _iptr(t), len(t), _iptr(b), len(b))
        if c == -1:
            raise MemoryError("not enough free KV blocks")
        if c < 0:
            raise ValueError("bad prompt or boundaries")
        return int(c)

    def append(self, ctx: int, token: int = 0):
        _check(self._lib.parrot_store_append(self._h, int(ctx), int(token)))

    def free(self, ctx: int):
        _check(self._lib.parrot_store_free(self._h, int(ctx)))

    @property
    def free_blocks(self) -> int:
        return int(self._lib.parrot_store_free_blocks(self._h))

    @property
    def num_prefixes(self) -> int:
        return int(self._lib.parrot_store_num_prefixes(self._h))

    def prefix_tokens(self, ctx: int) -> int:
        return int(self._lib.parrot_store_prefix_tokens(self._h, int(ctx)))

    def own_tokens(self, ctx: int) -> int:
        return int(self._lib.parrot_store_own_tokens(self._h, int(ctx)))

    def build_batch(self, ctxs: Sequence[int], pad_block: int = 0) -> Batch:
        c = _ints(ctxs)
        sh = BatchShape()
        _check(self._lib.parrot_store_batch_shape(self._h, _iptr(c), len(c), ctypes.byref(sh)))
        R, NG = len(c), sh.num_groups
        gid = np.zeros(R, np.int32)
        slen = np.zeros(R, np.int32)
        stab = np.zeros((R, sh.suffix_table_stride), np.int32)
        plen = np.zeros(max(NG, 1), np.int32)
        par = np.zeros(max(NG, 1), np.int32)
        ptab = np.zeros((max(NG, 1), sh.prefix_table_stride), np.int32)
        _check(self._lib.parrot_store_build_batch(
            self._h, _iptr(c), R, int(pad_block), _iptr(gid), _iptr(slen), _iptr(stab),
            _iptr(plen), _iptr(par), _iptr(ptab)))
        return Batch(gid, slen, stab, plen[:NG], par[:NG], ptab[:NG], sh)


__all__ = ["ContextStore", "Batch", "BatchShape", "ParrotError"]
