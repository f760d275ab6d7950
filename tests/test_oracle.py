"""The oracle against what the mathematics fixes (CPU only).

The pins live in ``oracle_pins``; this file runs each of them on the oracle
and then plants plausible mistakes in the oracle to show the pins catch them.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import oracle.attention as oa
import oracle_pins as pins
from oracle_pins import ALL_PINS, GOLDEN, PREFILL_PINS, pin_decomposition, tiny_paged_batch, decode_args


@pytest.mark.parametrize("name", sorted(ALL_PINS))
def test_oracle_pin(name):
    ALL_PINS[name](oracle.shared_prefix_decode)


def test_oracle_nested_decomposition():
    """Each chain level alone and the own tokens alone, merged, equal the
    whole nested context."""
    b = pins.tiny_nested_batch()
    p = b.plan
    whole = oracle.shared_prefix_decode(**pins.decode_args(b))
    for r in range(p.num_requests):
        parts = []
        for g in pins._walk_up(p.prefix_parents, int(p.group_ids[r])):
            gid = np.full_like(p.group_ids, -1)
            gid[r] = g
            parts.append(oracle.shared_prefix_decode(
                **pins.decode_args(b, group_ids=gid, suffix_lens=np.zeros_like(p.suffix_lens),
                                   prefix_parents=None), requests=[r]))
        if p.suffix_lens[r] > 0:
            parts.append(oracle.shared_prefix_decode(
                **pins.decode_args(b, group_ids=np.full_like(p.group_ids, -1)), requests=[r]))
        o, l = oracle.merge_segments([(x[0][0], x[1][0]) for x in parts])
        np.testing.assert_allclose(o, whole[0][r], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(l, whole[1][r], rtol=1e-13, atol=1e-13)


def test_oracle_decomposition_invariant():
    pin_decomposition(oracle.shared_prefix_decode, oracle.merge_segments)


def test_merge_worked_example():
    """Prefix-only and suffix-only results of the golden example merge exactly."""
    with open(os.path.join(GOLDEN, "worked_example.json")) as f:
        json.load(f)  # the derivation text states these four numbers
    o, l = oracle.merge_segments([(np.array([[2.0, 2.0]]), np.array([math.log(3)])),
                                  (np.array([[2.0, -2.0]]), np.array([math.log(3)]))])
    assert abs(l[0] - math.log(6)) < 1e-15
    assert np.allclose(o, [[2.0, 0.0]], atol=1e-15, rtol=0)


def test_merge_empty_segment_is_neutral():
    o1, l1 = np.array([[1.0, -2.0]]), np.array([0.3])
    empty = (np.zeros((1, 2)), np.array([-np.inf]))
    o, l = oracle.merge_segments([empty, (o1, l1), empty])
    assert np.array_equal(o, o1) and np.array_equal(l, l1)


def test_random_k_way_split_matches_whole():
    rng = np.random.default_rng(4)
    H, D, N = 3, 16, 300
    q = rng.standard_normal((H, D))
    K = rng.standard_normal((N, H, D))
    V = rng.standard_normal((N, H, D))
    o, l = oracle.attend(q, K, V, 0.25)
    for k in range(2, 9):
        cuts = np.sort(rng.choice(np.arange(1, N), size=k - 1, replace=False))
        bounds = [0, *cuts.tolist(), N]
        parts = [oracle.attend(q, K[a:b], V[a:b], 0.25) for a, b in zip(bounds, bounds[1:])]
        parts.append(oracle.attend(q, K[:0], V[:0], 0.25))   # an empty segment too
        mo, ml = oracle.merge_segments(parts)
        assert np.max(np.abs(mo - o)) < 1e-12
        assert np.max(np.abs(ml - l) / np.abs(l)) < 1e-13


def test_softmax_weights_sum_to_one():
    rng = np.random.default_rng(5)
    for N in (1, 2, 17, 1000):
        q = rng.standard_normal((4, 32)) * 3.0
        K = rng.standard_normal((N, 4, 32))
        V = rng.standard_normal((N, 4, 32))
        w = oracle.softmax_weights(q, K, 0.5)
        assert np.all(w >= 0)
        assert np.max(np.abs(w.sum(axis=1) - 1.0)) < 1e-12
        o, _ = oracle.attend(q, K, V, 0.5)
        assert np.max(np.abs(np.einsum("hn,nhd->hd", w, V) - o)) < 1e-12


def test_oracle_rejects_empty_context():
    b = tiny_paged_batch()
    args = decode_args(b, group_ids=np.full_like(b.plan.group_ids, -1),
                       suffix_lens=np.zeros_like(b.plan.suffix_lens))
    with pytest.raises(ValueError):
        oracle.shared_prefix_decode(**args)


# ------------------------------------------------------------ planted mistakes
def _mut_drop_last(monkeypatch):
    real = oa.request_kv

    def f(r, **kw):
        K, V = real(r, **kw)
        return K[:-1], V[:-1]
    monkeypatch.setattr(oa, "request_kv", f)


def _mut_gather_slot_shift(monkeypatch):
    def f(pool, table_row, length):
        B = int(pool.shape[2])
        rows = [oa.to_f64(pool[int(table_row[t // B]), :, (t + 1) % B, :]) for t in range(length)]
        H, D = int(pool.shape[1]), int(pool.shape[3])
        return np.stack(rows) if rows else np.zeros((0, H, D))
    monkeypatch.setattr(oa, "gather_sequence", f)


def _mut_gather_block_shift(monkeypatch):
    real = oa.gather_sequence

    def f(pool, table_row, length):
        row = np.asarray(table_row)
        return real(pool, np.concatenate([row[1:], row[:1]]) if len(row) > 1 else row, length)
    monkeypatch.setattr(oa, "gather_sequence", f)


def _mut_no_scale(monkeypatch):
    real = oa.attend
    monkeypatch.setattr(oa, "attend", lambda q, K, V, s: real(q, K, V, 1.0))


def _mut_lse_without_max(monkeypatch):
    def f(q, K, V, sm_scale):
        s = sm_scale * np.einsum("hd,nhd->hn", q, K)
        m = s.max(axis=1)
        z = np.log(np.exp(s - m[:, None]).sum(axis=1))
        w = np.exp(s - m[:, None] - z[:, None])
        return np.einsum("hn,nhd->hd", w, V), z
    monkeypatch.setattr(oa, "attend", f)


def _mut_kv_swapped(monkeypatch):
    real = oa.attend
    monkeypatch.setattr(oa, "attend", lambda q, K, V, s: real(q, V, K, s))


def _mut_sign(monkeypatch):
    real = oa.attend
    monkeypatch.setattr(oa, "attend", lambda q, K, V, s: real(q, K, V, -s))


def _mut_softmax_over_heads(monkeypatch):
    def f(q, K, V, sm_scale):
        s = sm_scale * np.einsum("hd,nhd->hn", q, K)
        m = s.max(axis=0)
        lse = m + np.log(np.exp(s - m[None, :]).sum(axis=0))
        w = np.exp(s - lse[None, :])
        return np.einsum("hn,nhd->hd", w, V), np.log(np.exp(s).sum(axis=1))
    monkeypatch.setattr(oa, "attend", f)


def _mut_wrong_group(monkeypatch):
    real = oa.request_kv

    def f(r, **kw):
        g = np.asarray(kw["group_ids"]).copy()
        ng = len(np.asarray(kw["prefix_lens"]))
        g = np.where(g >= 0, (g + 1) % max(ng, 1), g)
        kw = dict(kw, group_ids=g)
        return real(r, **kw)
    monkeypatch.setattr(oa, "request_kv", f)


def _mut_suffix_from_offset(monkeypatch):
    """Suffix read as if it continued the prefix's token numbering."""
    def f(r, *, prefix_k, prefix_v, suffix_k, suffix_v, prefix_tables, prefix_lens,
          suffix_tables, suffix_lens, group_ids, prefix_parents=None):
        g = int(np.asarray(group_ids)[r])
        S = int(np.asarray(suffix_lens)[r])
        P = int(np.asarray(prefix_lens)[g]) if g >= 0 else 0
        stab = np.asarray(suffix_tables)[r]
        B = int(suffix_k.shape[2])
        off = P % B
        Ks = oa.gather_sequence(suffix_k, stab, S + off)[off:]
        Vs = oa.gather_sequence(suffix_v, stab, S + off)[off:]
        if g < 0:
            return Ks, Vs
        ptab = np.asarray(prefix_tables)[g]
        return (np.concatenate([oa.gather_sequence(prefix_k, ptab, P), Ks]),
                np.concatenate([oa.gather_sequence(prefix_v, ptab, P), Vs]))
    monkeypatch.setattr(oa, "request_kv", f)


def _mut_head_shift(monkeypatch):
    real = oa.gather_sequence

    def f(pool, table_row, length):
        x = real(pool, table_row, length)
        return np.roll(x, 1, axis=1)
    monkeypatch.setattr(oa, "gather_sequence", f)


def _mut_prefix_ignored(monkeypatch):
    real = oa.request_kv

    def f(r, **kw):
        kw = dict(kw, group_ids=np.full_like(np.asarray(kw["group_ids"]), -1))
        K, V = real(r, **kw)
        if K.shape[0] == 0:
            return real(r, **dict(kw, suffix_lens=np.ones_like(np.asarray(kw["suffix_lens"]))))
        return K, V
    monkeypatch.setattr(oa, "request_kv", f)


def _mut_chain_leaf_only(monkeypatch):
    monkeypatch.setattr(oa, "group_chain", lambda g, parents=None: [g] if g >= 0 else [])


def _mut_chain_root_only(monkeypatch):
    real = oa.group_chain
    monkeypatch.setattr(oa, "group_chain", lambda g, parents=None: real(g, parents)[:1])


def _mut_chain_leaf_twice(monkeypatch):
    real = oa.group_chain

    def f(g, parents=None):
        c = real(g, parents)
        return c + c[-1:] if len(c) > 1 else c
    monkeypatch.setattr(oa, "group_chain", f)


def _mut_chain_skips_middle(monkeypatch):
    real = oa.group_chain

    def f(g, parents=None):
        c = real(g, parents)
        return [c[0], c[-1]] if len(c) > 2 else c
    monkeypatch.setattr(oa, "group_chain", f)


MUTANTS = {
    "drop_last_key": _mut_drop_last,
    "gather_slot_shift": _mut_gather_slot_shift,
    "gather_block_shift": _mut_gather_block_shift,
    "no_scale": _mut_no_scale,
    "lse_without_max": _mut_lse_without_max,
    "k_v_swapped": _mut_kv_swapped,
    "logit_sign": _mut_sign,
    "softmax_over_heads": _mut_softmax_over_heads,
    "wrong_group": _mut_wrong_group,
    "suffix_from_offset": _mut_suffix_from_offset,
    "head_shift": _mut_head_shift,
    "prefix_ignored": _mut_prefix_ignored,
    "chain_leaf_only": _mut_chain_leaf_only,
    "chain_root_only": _mut_chain_root_only,
    "chain_leaf_twice": _mut_chain_leaf_twice,
    "chain_skips_middle": _mut_chain_skips_middle,
}


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_catch_planted_mistake(mutant, monkeypatch):
    MUTANTS[mutant](monkeypatch)
    caught = []
    for name, pin in ALL_PINS.items():
        try:
            pin(oracle.shared_prefix_decode)
        except (AssertionError, ValueError, IndexError):
            caught.append(name)
    assert caught, f"no pin caught the planted mistake {mutant}"


# ------------------------------------------------------------------ prefill
@pytest.mark.parametrize("name", sorted(PREFILL_PINS))
def test_oracle_prefill_pin(name):
    PREFILL_PINS[name](oracle.shared_prefix_prefill)


def test_prefill_rejects_bad_offsets():
    batch, q, off = pins.tiny_prefill_case()
    args = pins.prefill_args(batch, q, off)
    bad = off.copy()
    bad[1] = bad[0] + int(batch.plan.suffix_lens[0]) + 1       # more rows than own tokens
    with pytest.raises(ValueError):
        oracle.shared_prefix_prefill(**dict(args, query_offsets=bad))
    with pytest.raises(ValueError):
        oracle.shared_prefix_prefill(**dict(args, q=q[:-1]))


def _positions_mutant(monkeypatch, f):
    real = oa.prefill_positions

    def g(query_offsets, suffix_lens):
        rows = real(query_offsets, suffix_lens)
        S = [int(x) for x in suffix_lens]
        qo = [int(x) for x in query_offsets]
        return [f(r, p, S, qo) for r, p in rows]
    monkeypatch.setattr(oa, "prefill_positions", g)


PREFILL_MUTANTS = {
    # a row does not see its own token
    "self_excluded": lambda mp: _positions_mutant(mp, lambda r, p, S, qo: (r, p - 1)),
    # a row sees the next own token too
    "next_included": lambda mp: _positions_mutant(mp, lambda r, p, S, qo: (r, min(p + 1, S[r] - 1))),
    # rows see every own token (no causal cut)
    "not_causal": lambda mp: _positions_mutant(mp, lambda r, p, S, qo: (r, S[r] - 1)),
    # rows numbered from the first own token instead of the last Q_r
    "positions_from_start": lambda mp: _positions_mutant(
        mp, lambda r, p, S, qo: (r, p - (S[r] - (qo[r + 1] - qo[r])))),
}


@pytest.mark.parametrize("mutant", sorted(PREFILL_MUTANTS))
def test_prefill_pins_catch_planted_mistake(mutant, monkeypatch):
    PREFILL_MUTANTS[mutant](monkeypatch)
    caught = []
    for name, pin in PREFILL_PINS.items():
        try:
            pin(oracle.shared_prefix_prefill)
        except (AssertionError, ValueError, IndexError):
            caught.append(name)
    assert caught, f"no pin caught the planted mistake {mutant}"


@pytest.mark.parametrize("mutant", ["prefix_ignored", "chain_leaf_only", "wrong_group",
                                    "gather_slot_shift", "lse_without_max"])
def test_prefill_pins_catch_shared_mistakes(mutant, monkeypatch):
    """Mistakes in the parts prefill shares with decode are caught by the
    prefill pins on their own."""
    MUTANTS[mutant](monkeypatch)
    caught = []
    for name, pin in PREFILL_PINS.items():
        if name == "prefill_last_row_is_decode":
            continue              # compares against the (equally mutated) decode
        try:
            pin(oracle.shared_prefix_prefill)
        except (AssertionError, ValueError, IndexError):
            caught.append(name)
    assert caught, f"no prefill pin caught the planted mistake {mutant}"
