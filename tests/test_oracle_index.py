"""Pins for the oracle's block index, insert, evict and match (CPU only).

* match: against a hash-free brute force -- c[r][i] = floor(max over prompts P placed on
  instance i of LCP(prompt_r, P) / B) -- the local prefix hit at block granularity of
  the paper's scoring template (Sec. 4.1) and reuse measurement (Sec. 3.1);
* insert / evict / dump: against a brute-force dictionary model of the entry set;
* the append-only invariant of agent sessions (Sec. 2): a turn extending a prompt placed
  on instance X matches every full block of that prompt on X.
"""
import math

import numpy as np
import pytest

import oracle

B = 16


def _streams(rng, n_streams, length, n_shared=0, shared_len=0):
    shared = rng.integers(0, 50, shared_len, dtype=np.int32)  # small vocab: many partial overlaps
    out = []
    for s in range(n_streams):
        body = rng.integers(0, 50, length, dtype=np.int32)
        if s < n_shared:
            body[:shared_len] = shared
        out.append(body)
    return out


def lcp(a, b):
    n = min(len(a), len(b))
    k = 0
    while k < n and a[k] == b[k]:
        k += 1
    return k


def _csr(prompts):
    off = np.zeros(len(prompts) + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in prompts])
    toks = np.concatenate(prompts).astype(np.int32) if prompts else np.zeros(0, np.int32)
    return toks, off


@pytest.mark.parametrize("seed", range(6))
def test_match_equals_bruteforce_lcp(seed):
    rng = np.random.default_rng(100 + seed)
    I = int(rng.integers(1, 6))
    streams = _streams(rng, 6, 200, n_shared=3, shared_len=int(rng.integers(0, 80)))
    # a few streams share token runs at random offsets too (partial overlaps mid-block)
    streams[4][:37] = streams[1][:37]
    placed = []  # (prompt, instance)
    for _ in range(12):
        s = int(rng.integers(0, len(streams)))
        placed.append((streams[s][: int(rng.integers(0, 200))], int(rng.integers(0, I))))
    queries = [streams[int(rng.integers(0, len(streams)))][: int(rng.integers(0, 200))] for _ in range(10)]
    queries.append(np.zeros(0, np.int32))

    ix = oracle.Index(10_000, I)
    toks, off = _csr([p for p, _ in placed])
    blk_off, keys = oracle.hash_blocks(toks, off, B, 42)
    assert ix.insert(keys, blk_off, [i for _, i in placed], list(range(len(placed))), 0) == 0
    qt, qo = _csr(queries)
    qb, qk = oracle.hash_blocks(qt, qo, B, 42)
    got = ix.match(qk, qb)
    for r, q in enumerate(queries):
        for i in range(I):
            best = max([lcp(q, p) for p, inst in placed if inst == i], default=0)
            assert got[r, i] == best // B, (r, i)


class DictIndex:
    """Brute-force model: {(key, inst): [session, epoch]}."""

    def __init__(self, capacity, I):
        self.cap, self.I, self.d, self.status = capacity, I, {}, 0

    def insert(self, keys, blk_off, inst, sess, epoch):
        pairs = [(int(keys[b]), int(inst[r]), int(sess[r])) for r in range(len(blk_off) - 1)
                 for b in range(blk_off[r], blk_off[r + 1])]
        fresh = {(k, i) for k, i, _ in pairs if (k, i) not in self.d}
        if len(self.d) + len(fresh) > self.cap:
            self.status = self.status or -2
            return -2
        for k, i, s in pairs:
            if (k, i) in self.d:
                self.d[(k, i)][1] = max(self.d[(k, i)][1], epoch)
            else:
                self.d[(k, i)] = [s, epoch]
        return 0

    def evict(self, num, den):
        m = math.ceil(len(self.d) * num / den)
        order = sorted(self.d, key=lambda ki: (self.d[ki][1], ki[0], ki[1]))
        for ki in order[:m]:
            del self.d[ki]

    def dump(self):
        items = sorted(self.d.items())
        keys = np.array([k for (k, _), _ in items], np.uint64)
        vals = np.array([(i << 48) | (e << 24) | s for (_, i), (s, e) in items], np.uint64)
        return keys, vals


def _random_batches(rng, I, n_batches, R, maxlen):
    streams = _streams(rng, 8, maxlen, n_shared=4, shared_len=64)
    out = []
    for e in range(n_batches):
        prompts = [streams[int(rng.integers(0, 8))][: int(rng.integers(0, maxlen))] for _ in range(R)]
        toks, off = _csr(prompts)
        blk_off, keys = oracle.hash_blocks(toks, off, B, 9)
        inst = rng.integers(0, I, R).astype(np.int32)
        sess = rng.integers(0, 1000, R).astype(np.uint32)
        out.append((keys, blk_off, inst, sess, e))
    return out


@pytest.mark.parametrize("seed", range(4))
def test_insert_evict_dump_equal_dictionary_model(seed):
    rng = np.random.default_rng(200 + seed)
    I = 4
    ix, model = oracle.Index(10_000, I), DictIndex(10_000, I)
    for keys, blk_off, inst, sess, e in _random_batches(rng, I, 6, 9, 300):
        assert ix.insert(keys, blk_off, inst, sess, e) == model.insert(keys, blk_off, inst, sess, e) == 0
        k1, v1 = ix.dump()
        k2, v2 = model.dump()
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)
        if e % 2:
            n_before = ix.size
            ix.evict(1, 20)
            model.evict(1, 20)
            assert ix.size == n_before - math.ceil(n_before / 20)
            k1, v1 = ix.dump()
            k2, v2 = model.dump()
            assert np.array_equal(k1, k2) and np.array_equal(v1, v2)


def test_duplicate_pairs_take_lowest_request_session_and_max_epoch():
    ix = oracle.Index(100, 3)
    keys = np.array([11, 12, 11, 12, 13], np.uint64)
    blk_off = np.array([0, 2, 4, 5])
    assert ix.insert(keys, blk_off, [1, 1, 2], [70, 80, 90], 5) == 0
    assert ix.insert([11], [0, 1], [1], [99], 3) == 0  # older epoch: epoch stays 5, session stays 70
    k, v = ix.dump()
    inst, ep, se = oracle.unpack_vals(v)
    assert list(zip(k.tolist(), inst.tolist(), ep.tolist(), se.tolist())) == [
        (11, 1, 5, 70), (12, 1, 5, 70), (13, 2, 5, 90)]


def test_efull_and_einval_leave_index_unchanged():
    ix = oracle.Index(3, 2)
    assert ix.insert([5, 6], [0, 2], [0], [1], 0) == 0
    before = ix.dump()
    assert ix.insert([7, 8], [0, 2], [1], [2], 1) == oracle.EFULL  # 2 + 2 > 3
    assert ix.status == oracle.EFULL
    assert all(np.array_equal(a, b) for a, b in zip(before, ix.dump()))
    # refreshing existing entries plus one new fits exactly
    assert ix.insert([5, 6, 9], [0, 3], [0], [3], 2) == 0
    assert ix.size == 3
    for bad in (dict(keys=[0], inst=[0], sess=[1]), dict(keys=[2**64 - 1], inst=[0], sess=[1]),
                dict(keys=[4], inst=[2], sess=[1]), dict(keys=[4], inst=[0], sess=[1 << 24])):
        j = oracle.Index(10, 2)
        assert j.insert(bad["keys"], [0, 1], bad["inst"], bad["sess"], 0) == oracle.EINVAL
        assert j.size == 0 and j.status == oracle.EINVAL
    j = oracle.Index(10, 2)
    assert j.insert([4, 5], [0, 2, 1], [0, 0], [1, 1], 0, n_blocks=2) == oracle.EINVAL  # decreasing range
    assert j.insert([4, 5], [0, 2, 2], [0, 0], [1, 1], 0) == 0  # an empty request with any range is fine
    assert j.insert([4], [0, 1], [0], [1], 1 << 22) == oracle.EINVAL  # epoch out of range (host check)


def test_evict_exact_count_and_order():
    ix, model = oracle.Index(1000, 2), DictIndex(1000, 2)
    rng = np.random.default_rng(3)
    for e in range(5):
        keys = rng.integers(1, 2**63, 40, dtype=np.uint64)
        blk_off = np.array([0, 20, 40])
        for m in (ix, model):
            m.insert(keys, blk_off, [0, 1], [e, e], e)
    for num, den in ((1, 20), (1, 3), (0, 5), (7, 7)):
        n = ix.size
        ix.evict(num, den)
        model.evict(num, den)
        assert ix.size == n - math.ceil(n * num / den)
        assert all(np.array_equal(a, b) for a, b in zip(ix.dump(), model.dump()))
    assert ix.evict(1, 0) == oracle.EINVAL and ix.evict(3, 2) == oracle.EINVAL


def test_match_first_miss_after_eviction():
    """With entries evicted in (epoch, key, instance) order a descendant block can outlive
    its parent; the match must stop at the first missing block for each instance."""
    rng = np.random.default_rng(8)
    I = 3
    streams = _streams(rng, 5, 400, n_shared=3, shared_len=100)
    ix = oracle.Index(100_000, I)
    prefix_of_key = {}
    placed = set()  # (token-prefix tuple, inst) whose key is in the index
    for e in range(4):
        prompts = [streams[int(rng.integers(0, 5))][: int(rng.integers(50, 400))] for _ in range(6)]
        toks, off = _csr(prompts)
        blk_off, keys = oracle.hash_blocks(toks, off, B, 1)
        inst = rng.integers(0, I, 6).astype(np.int32)
        for r, p in enumerate(prompts):
            for j in range(len(p) // B):
                prefix_of_key[int(keys[blk_off[r] + j])] = tuple(p[: B * (j + 1)].tolist())
        ix.insert(keys, blk_off, inst, np.arange(6), e)
        ix.evict(1, 4)
    k, v = ix.dump()
    inst, _, _ = oracle.unpack_vals(v)
    placed = {(prefix_of_key[int(kk)], int(ii)) for kk, ii in zip(k, inst)}
    queries = [streams[s][:400] for s in range(5)]
    qt, qo = _csr(queries)
    qb, qk = oracle.hash_blocks(qt, qo, B, 1)
    got = ix.match(qk, qb)
    saw_orphan = False
    for r, q in enumerate(queries):
        for i in range(I):
            j = 0
            while j < len(q) // B and (tuple(q[: B * (j + 1)].tolist()), i) in placed:
                j += 1
            assert got[r, i] == j
            later = any((tuple(q[: B * (jj + 1)].tolist()), i) in placed for jj in range(j + 1, len(q) // B))
            saw_orphan |= later
    assert saw_orphan  # the case exercises a descendant that outlived its parent


def test_append_only_turn_matches_previous_prompt_on_its_instance():
    rng = np.random.default_rng(9)
    I, S = 6, 20
    streams = [rng.integers(0, 151936, 3000, dtype=np.int32) for _ in range(S)]
    lens0 = rng.integers(100, 1500, S)
    lens1 = lens0 + rng.integers(1, 1500, S)
    home = rng.integers(0, I, S).astype(np.int32)
    ix = oracle.Index(100_000, I)
    t0, o0 = _csr([streams[s][: lens0[s]] for s in range(S)])
    b0, k0 = oracle.hash_blocks(t0, o0, B, 5)
    ix.insert(k0, b0, home, np.arange(S), 0)
    t1, o1 = _csr([streams[s][: lens1[s]] for s in range(S)])
    b1, k1 = oracle.hash_blocks(t1, o1, B, 5)
    c = ix.match(k1, b1)
    for s in range(S):
        assert c[s, home[s]] == lens0[s] // B
        assert all(c[s, i] == 0 for i in range(I) if i != home[s])


def test_match_bad_range_gives_zero_row_and_einval():
    ix = oracle.Index(10, 2)
    ix.insert([5, 6], [0, 2], [1], [1], 0)
    c = ix.match(np.array([5, 6], np.uint64), np.array([0, 2, 1]), n_blocks=2)
    assert c.tolist() == [[0, 2], [0, 0]]
    assert ix.last_rc == oracle.EINVAL and ix.status == oracle.EINVAL
