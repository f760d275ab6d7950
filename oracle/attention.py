"""Plain float64 decode attention over a paged KV cache (test infrastructure).

Definitions (Section 5.3 and the "Kernel Optimization" paragraph of Section 7;
the paper builds on the softmax attention of FlashAttention and PagedAttention
and does not restate it, so the standard definition is written out here):

  For request r and head h, with g = group_ids[r], P = prefix_lens[g] (P = 0
  when g = -1) and S = suffix_lens[r], the keys are
      K_j = prefix key j of group g         for 0 <= j < P
      K_j = suffix key (j - P) of request r for P <= j < P + S
  (values likewise), and
      s_j    = sm_scale * sum_d q[r,h,d] * K_j[d]
      m      = max_j s_j
      lse    = m + ln sum_j exp(s_j - m)
      w_j    = exp(s_j - lse)
      out[d] = sum_j w_j * V_j[d]

  Paged storage (Section 7, the per-request page table kept from
  PagedAttention): token t of a sequence with block table row ``tbl`` lives at
  pool[tbl[t // B], h, t % B, :] of a [num_blocks, H, B, D] pool.

  Nested prefixes: a prompt can share prefixes at several depths (a prefix
  hash is taken after every semantic variable, Section 5.3, and a context can
  be forked from a forked context through parent_context_id, Section 7).  With
  prefix_parents[g] naming the group whose prefix precedes group g's (-1 for
  none), a request of group g reads the prefixes of g's ancestors, outermost
  first, then g's own prefix, then its own tokens.  Without prefix_parents
  every group stands alone.

  Prefill of a forked context (Section 7, Fill with a parent_context_id: the
  new prompt tokens of a context forked from a parent are filled on top of the
  parent's KV cache, so only the new tokens are computed).  Request r brings
  Q_r <= S_r new rows, its last Q_r own tokens, stacked in request order:
  row query_offsets[r] + j is own position p = S_r - Q_r + j.  Its keys are
  those of the decode case cut after own token p: the prefixes of its group's
  chain, then own tokens 0..p (the usual causal self-attention of a decoder,
  which the paper takes as given).  With Q_r = S_r = 1 it is one decode step.

All inputs are upcast exactly to float64 before any arithmetic.
"""
from __future__ import annotations

from typing import Iterable, Optional, Sequence

import numpy as np

try:  # torch is only needed to read bfloat16 / float16 tensors exactly
    import torch
except ImportError:  # pragma: no cover
    torch = None


def to_f64(x) -> np.ndarray:
    """Exact upcast of a numpy array or torch CPU tensor to float64."""
    if torch is not None and isinstance(x, torch.Tensor):
        return x.detach().to("cpu", torch.float64).numpy()
    return np.asarray(x, dtype=np.float64)


def _ints(x) -> np.ndarray:
    if torch is not None and isinstance(x, torch.Tensor):
        x = x.detach().cpu().numpy()
    return np.asarray(x, dtype=np.int64)


def gather_sequence(pool, table_row: Sequence[int], length: int) -> np.ndarray:
    """Tokens 0..length-1 of one paged sequence as float64 [length, H, D].

    Token t is pool[table_row[t // B], :, t % B, :] (Section 7, paged KV with a
    per-request page table).
    """
    B = int(pool.shape[2])
    H, D = int(pool.shape[1]), int(pool.shape[3])
    if length == 0:
        return np.zeros((0, H, D), dtype=np.float64)
    nblk = -(-length // B)
    blocks = _ints(table_row)[:nblk]
    x = to_f64(pool[blocks])                       # [nblk, H, B, D]
    x = x.transpose(0, 2, 1, 3).reshape(nblk * B, H, D)
    return x[:length]


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, sm_scale: float):
    """Softmax attention of one query per head over N keys.

    q: [H, D], K, V: [N, H, D] (float64).  Returns (out [H, D], lse [H]).
    An empty key set gives out = 0 and lse = -inf (the neutral element of
    ``merge_segments``).
    """
    H, D = q.shape
    if K.shape[0] == 0:
        return np.zeros((H, D)), np.full(H, -np.inf)
    s = sm_scale * np.einsum("hd,nhd->hn", q, K)   # [H, N]
    m = s.max(axis=1)
    lse = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
    w = np.exp(s - lse[:, None])
    out = np.einsum("hn,nhd->hd", w, V)
    return out, lse


def softmax_weights(q: np.ndarray, K: np.ndarray, sm_scale: float) -> np.ndarray:
    """The weights w_j of ``attend`` as [H, N]."""
    s = sm_scale * np.einsum("hd,nhd->hn", q, K)
    m = s.max(axis=1)
    lse = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
    return np.exp(s - lse[:, None])


def merge_segments(parts: Iterable[tuple]) -> tuple:
    """Combine attention results of disjoint key segments.

    For segments i with results (o_i, l_i) computed by ``attend`` on each
    segment alone, attention over their union is
        l = ln sum_i exp(l_i),   o = sum_i exp(l_i - l) * o_i,
    which is how the paper's kernel joins the prefix's interim results with
    the non-shared tokens (Section 7, "Kernel Optimization").  Empty segments
    (l_i = -inf) carry weight zero.
    """
    parts = list(parts)
    ls = np.stack([p[1] for p in parts])            # [k, H]
    os_ = np.stack([p[0] for p in parts])           # [k, H, D]
    m = ls.max(axis=0)
    m_safe = np.where(np.isfinite(m), m, 0.0)
    wsum = np.exp(ls - m_safe).sum(axis=0)
    l = m_safe + np.log(wsum)
    w = np.exp(ls - np.where(np.isfinite(l), l, 0.0))   # [k, H]
    o = np.einsum("kh,khd->hd", w, os_)
    return o, l


def group_chain(g: int, prefix_parents=None) -> list:
    """The groups whose prefixes a request of group g reads, outermost first."""
    if g < 0:
        return []
    if prefix_parents is None:
        return [g]
    parents = _ints(prefix_parents)
    chain = [g]
    while parents[chain[-1]] >= 0:
        if len(chain) > len(parents):
            raise ValueError("prefix_parents contains a cycle")
        chain.append(int(parents[chain[-1]]))
    return chain[::-1]


def request_kv(r: int, *, prefix_k, prefix_v, suffix_k, suffix_v,
               prefix_tables, prefix_lens, suffix_tables, suffix_lens, group_ids,
               prefix_parents=None):
    """Keys and values of request r: the prefixes of its group's chain, then
    its own suffix."""
    g = int(_ints(group_ids)[r])
    S = int(_ints(suffix_lens)[r])
    stab = _ints(suffix_tables)[r]
    Ks = [gather_sequence(suffix_k, stab, S)]
    Vs = [gather_sequence(suffix_v, stab, S)]
    Kp, Vp = [], []
    for a in group_chain(g, prefix_parents):
        P = int(_ints(prefix_lens)[a])
        ptab = _ints(prefix_tables)[a]
        Kp.append(gather_sequence(prefix_k, ptab, P))
        Vp.append(gather_sequence(prefix_v, ptab, P))
    return np.concatenate(Kp + Ks), np.concatenate(Vp + Vs)


def shared_prefix_decode(q, prefix_k, prefix_v, suffix_k, suffix_v, prefix_tables,
                         prefix_lens, suffix_tables, suffix_lens, group_ids,
                         sm_scale: float, requests: Optional[Sequence[int]] = None,
                         prefix_parents=None):
    """Naive per-request decode attention over concat(prefixes, suffix).

    Returns (out [n, H, D], lse [n, H]) in float64 for the requests listed in
    ``requests`` (all requests, in order, by default).
    """
    qf = to_f64(q)
    R, H, D = qf.shape
    if requests is None:
        requests = range(R)
    requests = list(requests)
    out = np.zeros((len(requests), H, D))
    lse = np.zeros((len(requests), H))
    for i, r in enumerate(requests):
        K, V = request_kv(r, prefix_k=prefix_k, prefix_v=prefix_v, suffix_k=suffix_k,
                          suffix_v=suffix_v, prefix_tables=prefix_tables,
                          prefix_lens=prefix_lens, suffix_tables=suffix_tables,
                          suffix_lens=suffix_lens, group_ids=group_ids,
                          prefix_parents=prefix_parents)
        if K.shape[0] == 0:
            raise ValueError(f"request {r} has an empty context")
        out[i], lse[i] = attend(qf[r], K, V, sm_scale)
    return out, lse


def prefill_positions(query_offsets, suffix_lens) -> list:
    """(request, own position) of every query row, in row order."""
    qo = _ints(query_offsets)
    S = _ints(suffix_lens)
    if qo.shape[0] != S.shape[0] + 1 or qo[0] != 0:
        raise ValueError("query_offsets must hold R + 1 entries starting at 0")
    rows = []
    for r in range(S.shape[0]):
        Q = int(qo[r + 1] - qo[r])
        if Q < 0 or Q > S[r]:
            raise ValueError(f"request {r}: {Q} query rows for {S[r]} own tokens")
        rows += [(r, int(S[r]) - Q + j) for j in range(Q)]
    return rows


def shared_prefix_prefill(q, query_offsets, prefix_k, prefix_v, suffix_k, suffix_v,
                          prefix_tables, prefix_lens, suffix_tables, suffix_lens, group_ids,
                          sm_scale: float, rows: Optional[Sequence[int]] = None,
                          prefix_parents=None):
    """Naive per-row prefill attention: row i of request r at own position p
    attends to r's prefix chain and its own tokens 0..p.

    q: [T, H, D] query rows (T = query_offsets[R]).  Returns (out [n, H, D],
    lse [n, H]) in float64 for the rows listed in ``rows`` (all by default).
    """
    qf = to_f64(q)
    pos = prefill_positions(query_offsets, suffix_lens)
    if len(pos) != qf.shape[0]:
        raise ValueError(f"{qf.shape[0]} query rows, offsets describe {len(pos)}")
    rows = list(range(len(pos)) if rows is None else rows)
    H, D = qf.shape[1], qf.shape[2]
    out = np.zeros((len(rows), H, D))
    lse = np.zeros((len(rows), H))
    kv = {}
    gid = _ints(group_ids)
    plen = _ints(prefix_lens)
    for i, t in enumerate(rows):
        r, p = pos[t]
        if r not in kv:
            kv[r] = request_kv(r, prefix_k=prefix_k, prefix_v=prefix_v, suffix_k=suffix_k,
                               suffix_v=suffix_v, prefix_tables=prefix_tables,
                               prefix_lens=prefix_lens, suffix_tables=suffix_tables,
                               suffix_lens=suffix_lens, group_ids=group_ids,
                               prefix_parents=prefix_parents)
        K, V = kv[r]
        n_prefix = sum(int(plen[a]) for a in group_chain(int(gid[r]), prefix_parents))
        n = n_prefix + p + 1
        out[i], lse[i] = attend(qf[t], K[:n], V[:n], sm_scale)
    return out, lse

