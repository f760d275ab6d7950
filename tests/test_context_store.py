"""The host-side context store (CPU): prefix sharing at semantic-variable
boundaries, block accounting, and the batch arrays it emits, checked against
a plain Python model of the same rules."""
import numpy as np
import pytest

from paper_2405_19888_amd.context import ContextStore


class Model:
    """Reference: cached prefixes are the token tuples tokens[:b] at every
    boundary b of every live context; a context reads its deepest one."""

    def __init__(self, B):
        self.B = B
        self.ctx = {}            # id -> (boundary prefixes as tuples, own tokens)

    def fill(self, cid, tokens, bounds):
        prefixes = [tuple(tokens[:b]) for b in bounds]
        own = len(tokens) - (bounds[-1] if bounds else 0)
        self.ctx[cid] = (prefixes, own)

    def cached(self):
        return {p for prefixes, _ in self.ctx.values() for p in prefixes}

    def blocks_used(self):
        used = 0
        cached = sorted(self.cached(), key=len)
        for p in cached:
            parent = max((q for q in cached if len(q) < len(p) and p[:len(q)] == q), key=len,
                         default=())
            used += -(-(len(p) - len(parent)) // self.B)
        return used + sum(-(-own // self.B) for _, own in self.ctx.values())


SEGMENTS = [[1, 2, 3] * 7, [4, 5] * 9, [9] * 16, [6, 7, 8, 9, 10], [11] * 33, [12, 13]]


def random_prompt(rng):
    """Prompts built from a few shared segments, so prefixes repeat."""
    k = int(rng.integers(0, 4))
    segs = [SEGMENTS[int(rng.integers(0, len(SEGMENTS)))] for _ in range(k)]
    tokens, bounds = [], []
    for s in segs:
        tokens += s
        bounds.append(len(tokens))
    tokens += rng.integers(100, 200, size=int(rng.integers(0 if k else 1, 40))).tolist()
    if bounds and bounds[-1] == len(tokens) and rng.random() < 0.5:
        pass                                  # prompt ends on a boundary: no own tokens
    return tokens, bounds


def check_batch(st, model, ids):
    b = st.build_batch(ids, pad_block=st.num_blocks)
    B = st.block_size
    seen = {}
    for i, c in enumerate(ids):
        prefixes, own = model.ctx[c]
        assert b.suffix_lens[i] == own == st.own_tokens(c)
        # the chain of groups holds the context's boundary prefixes, outermost first
        chain, g = [], int(b.group_ids[i])
        while g >= 0:
            chain.insert(0, g)
            assert b.prefix_parents[g] < g
            g = int(b.prefix_parents[g])
        lens = [len(p) for p in prefixes]
        assert [int(sum(b.prefix_lens[x] for x in chain[:j + 1])) for j in range(len(chain))] == lens
        assert st.prefix_tokens(c) == (lens[-1] if lens else 0)
        nown = -(-own // B)
        row = b.suffix_tables[i]
        assert np.all(row[nown:] == st.num_blocks)
        for blk in row[:nown]:
            assert seen.setdefault(int(blk), ("own", c)) == ("own", c)
    for g in range(b.shape.num_groups):
        n = -(-int(b.prefix_lens[g]) // B)
        for blk in b.prefix_tables[g][:n]:
            assert seen.setdefault(int(blk), ("prefix", g)) == ("prefix", g)
        assert np.all(b.prefix_tables[g][n:] == st.num_blocks)
    return b


def test_shared_system_prompt_two_levels():
    st = ContextStore(block_size=16, num_blocks=100)
    sysp = list(range(1, 41))                 # 40 tokens: 3 blocks
    fs1, fs2 = [50] * 20, [60] * 20
    a = st.fill(sysp + fs1 + [7, 8], [40, 60])
    b = st.fill(sysp + fs1 + [9], [40, 60])
    c = st.fill(sysp + fs2, [40, 60])
    d = st.fill(sysp + [1, 2, 3], [40])
    assert st.num_prefixes == 3               # system prompt and two few-shot blocks
    assert st.free_blocks == 100 - (3 + 2 + 2) - 3
    batch = st.build_batch([a, b, c, d])
    assert batch.shape.num_groups == 3 and batch.shape.max_prefix_depth == 2
    assert batch.shape.max_group_size == 4
    assert list(batch.prefix_lens) == [40, 20, 20] and list(batch.prefix_parents) == [-1, 0, 0]
    assert batch.group_ids[0] == batch.group_ids[1] != batch.group_ids[2]
    assert batch.group_ids[3] == 0
    assert list(batch.suffix_lens) == [2, 1, 0, 3]
    for x in (a, b, c, d):
        st.free(x)
    assert st.free_blocks == 100 and st.num_prefixes == 0


def test_same_hash_path_different_tokens_do_not_share():
    st = ContextStore(block_size=4, num_blocks=64)
    a = st.fill([1, 2, 3, 4, 5], [4])
    b = st.fill([1, 2, 3, 5, 5], [4])
    assert st.num_prefixes == 2
    batch = st.build_batch([a, b])
    assert batch.group_ids[0] != batch.group_ids[1]


def test_out_of_blocks_changes_nothing():
    st = ContextStore(block_size=16, num_blocks=4)
    a = st.fill(list(range(40)), [32])        # 2 + 1 blocks
    with pytest.raises(MemoryError):
        st.fill(list(range(40)) + [1] * 40, [32, 72])   # needs 2 (new segment) + 1 own
    assert st.free_blocks == 1 and st.num_prefixes == 1
    st.append(a)
    for _ in range(7):
        st.append(a)
    assert st.own_tokens(a) == 16 and st.free_blocks == 1
    st.append(a)                              # token 17 opens the last free block
    assert st.free_blocks == 0
    with pytest.raises(Exception):
        for _ in range(16):
            st.append(a)
    st.free(a)
    assert st.free_blocks == 4 and st.num_prefixes == 0


def test_bad_arguments():
    st = ContextStore(block_size=16, num_blocks=8)
    with pytest.raises(ValueError):
        st.fill([], [])
    with pytest.raises(ValueError):
        st.fill([1, 2, 3], [2, 2])
    with pytest.raises(ValueError):
        st.fill([1, 2, 3], [4])
    with pytest.raises(Exception):
        st.free(3)
    with pytest.raises(Exception):
        st.build_batch([5])


@pytest.mark.parametrize("seed", range(6))
def test_random_operations_match_model(seed):
    rng = np.random.default_rng(seed)
    B = [4, 16][seed % 2]
    st = ContextStore(block_size=B, num_blocks=400)
    model = Model(B)
    live = []
    for step in range(150):
        op = rng.random()
        if op < 0.5 or not live:
            tokens, bounds = random_prompt(rng)
            try:
                c = st.fill(tokens, bounds)
            except MemoryError:
                assert model.blocks_used() + 1 > 0
                continue
            model.fill(c, tokens, bounds)
            live.append(c)
        elif op < 0.8:
            c = live[int(rng.integers(0, len(live)))]
            try:
                st.append(c)
            except Exception:
                continue
            p, own = model.ctx[c]
            model.ctx[c] = (p, own + 1)
        else:
            c = live.pop(int(rng.integers(0, len(live))))
            st.free(c)
            del model.ctx[c]
        assert st.num_prefixes == len(model.cached())
        assert st.free_blocks == 400 - model.blocks_used()
        if live and step % 10 == 0:
            check_batch(st, model, live)
    for c in live:
        st.free(c)
    assert st.free_blocks == 400 and st.num_prefixes == 0
