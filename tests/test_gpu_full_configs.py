"""Configurations 1-3 at their full sizes on the GPU, in the launch configuration bench.py
times (hash + partition in one call, the region-ordered lookup, match, route).

The oracle cannot hold these indexes, so each test runs the configuration open loop --
every turn but the last entered on a seeded random placement -- and checks a sample of the
last batch's requests bit for bit: their block keys, matched rows, targets and branches,
against the oracle run on the exact restriction of the index to their keys.  For a
sampled request that restriction is its own session's earlier turns (each a prefix of its
prompt) on their placements, plus its shared system prefix on every instance that
received a turn starting with that prefix; no other entry carries one of its keys (other
sessions' private blocks are chained from different tokens).  Configuration 4 is checked
the same way by bench.py at full size, configuration 0 in full in test_gpu_parity.
After the check the last batch is entered at its targets through the product path's
insert (smetric_index_insert_probed) and checked at full size by what that insert must
satisfy on an index that is prefix-closed on every instance: the entry count grows by
exactly the distinct new (key, target) pairs, and every request then sees its whole
prompt on its target (append-only prompts, Sec. 2; the target caches what it prefills,
Sec. 4.2).  Configuration 3 then runs one 5 % eviction of its full index, checked by
what eviction must satisfy at any size: exactly ceil(N/20) entries leave, and every one that leaves
precedes every one that stays under (epoch, key, instance)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_08565_amd import workload as W
from tests.parity import check_probed_insert_full, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def _csr(parts):
    off = np.zeros(len(parts) + 1, np.int64)
    off[1:] = np.cumsum([len(p) for p in parts])
    return (np.concatenate(parts) if parts else np.zeros(0, parts[0].dtype)), off


def _open_loop_last_batch(wl, capacity, n_sample, seed):
    """Enter turns 0 .. T-2 on their placements, run the last batch; returns what the
    checks need."""
    from paper_2607_08565_amd import smetric as S
    T, I = wl.n_turns, wl.n_inst
    place = W.open_loop_placement(wl)
    gix = S.Index(capacity, I)
    for t in range(T - 1):
        b = wl.batch(t)
        blk_off, nb = S.block_offsets(b.tok_off)
        d_boff = to_dev(blk_off)
        keys = S.hash_blocks(to_dev(b.tokens), to_dev(b.tok_off), d_boff, nb)
        gix.insert(keys, d_boff, nb, to_dev(place[t]), to_dev(np.arange(wl.n_sess, dtype=np.uint32)), t)
        del keys
        n, st = gix.stats()
        assert st == 0, f"turn {t}: status {st}"
        say(f"  turn {t} entered: {nb} blocks, {n} entries")
    b = wl.batch(T - 1, place[T - 2])
    blk_off, nb = S.block_offsets(b.tok_off)
    d_boff = to_dev(blk_off)
    keys, state = gix.hash_partition(to_dev(b.tokens), to_dev(b.tok_off), d_boff, nb)
    gix.probe_lookup(state, keys, d_boff, nb)
    gm = gix.match_probed(state, keys, d_boff, nb)
    gt, gb = S.route(gm, to_dev(b.prompt_len), to_dev(b.hist_len), to_dev(b.turn), to_dev(b.q), W.DEFAULT_PARAMS,
                     b.rr_base)
    say(f"  last batch: {b.n_req} requests, {nb} blocks, {b.n_tokens} tokens")
    sample = np.sort(np.random.default_rng(seed).choice(wl.n_sess, n_sample, replace=False))
    return dict(gix=gix, place=place, batch=b, blk_off=blk_off, keys=keys, state=state, nb=nb,
                gm=gm.cpu().numpy(), gt=gt.cpu().numpy(), gb=gb.cpu().numpy(), sample=sample)


def _check_insert(run):
    """The product path's insert of the last batch at its targets, checked at full size."""
    check_probed_insert_full(run["gix"], run["batch"], run["blk_off"], run["nb"], run["keys"], run["state"],
                             run["gm"], run["gt"])


def _check_sample(wl, run, capacity):
    T, I, P = wl.n_turns, wl.n_inst, W.prefix_blocks(wl.cfg)
    b, place, sample = run["batch"], run["place"], run["sample"]
    toks, toff = _csr([wl.streams[s][: wl.lens[T - 1, s]] for s in sample])
    ob, ok = oracle.hash_blocks(toks, toff, W.BLOCK, W.DEFAULT_SEED)
    gkeys = run["keys"].cpu().numpy()
    for i, s in enumerate(sample):
        g = gkeys[run["blk_off"][s]: run["blk_off"][s + 1]]
        assert np.array_equal(g, ok[ob[i]: ob[i + 1]]), f"keys of request {s}"
    # the restriction: own earlier turns, and each sampled prefix on every instance that got it
    segs, inst = [], []
    for i, s in enumerate(sample):
        mine = ok[ob[i]: ob[i + 1]]
        for t in range(T - 1):
            segs.append(mine[: wl.lens[t, s] // W.BLOCK])
            inst.append(place[t, s])
    for p in np.unique(wl.prefix_of[sample]):
        i = int(np.nonzero(wl.prefix_of[sample] == p)[0][0])
        pkeys = ok[ob[i]: ob[i] + P]
        holders = np.unique(place[: T - 1][:, wl.prefix_of == p])
        for h in holders:
            segs.append(pkeys)
            inst.append(h)
    rk, roff = _csr(segs)
    oix = oracle.Index(capacity, I)
    assert oix.insert(rk, roff, np.asarray(inst, np.int32), np.zeros(len(segs), np.uint32), 0) == 0
    say(f"  restricted oracle index: {oix.size} entries for {len(sample)} sampled requests")
    om = oix.match(ok, ob)
    for i, s in enumerate(sample):
        assert np.array_equal(run["gm"][s], om[i]), f"matched row of request {s}"
        ot, obr = oracle.route(om[i: i + 1], b.prompt_len[s: s + 1], b.hist_len[s: s + 1], b.turn[s: s + 1], b.q,
                               W.DEFAULT_PARAMS, b.rr_base + int(s))
        assert run["gt"][s] == ot[0] and run["gb"][s] == obr[0], f"decision of request {s}"
    return np.bincount(run["gb"][sample], minlength=5)


def test_config1_full_size_sampled():
    """4,096 sessions x 10 turns on 64 instances, 16 Zipf(1.1) 2,048-token prefixes."""
    wl = W.config1()
    run = _open_loop_last_batch(wl, 45_000_000, 24, 101)
    br = _check_sample(wl, run, 45_000_000)
    _check_insert(run)
    say("  sampled branches", br.tolist(), "all branches", np.bincount(run["gb"], minlength=5).tolist())


def test_config2_full_size_sampled():
    """1,024 sessions x 30 turns on 256 instances, prompts up to 131,072 tokens."""
    wl = W.config2()
    run = _open_loop_last_batch(wl, 160_000_000, 12, 102)
    br = _check_sample(wl, run, 160_000_000)
    _check_insert(run)
    say("  sampled branches", br.tolist(), "all branches", np.bincount(run["gb"], minlength=5).tolist())


def test_config3_full_size_sampled_and_eviction():
    """8,192 sessions sharing one 32,768-token prefix on 128 instances; then one 5 % LRU
    eviction of the whole index."""
    wl = W.config3()
    cap = 72_000_000  # a 0.7 load factor of ~50M entries
    run = _open_loop_last_batch(wl, cap, 16, 103)
    _check_sample(wl, run, cap)
    _check_insert(run)
    gix = run["gix"]
    k0, v0 = gix.dump()
    gix.evict(1, 20)
    k1, v1 = gix.dump()
    n0, n1 = len(k0), len(k1)
    assert n0 - n1 == -(-n0 // 20), f"evicted {n0 - n1} of {n0}"
    # survivors: entries of the first dump whose (key, instance) is in the second, found by
    # sorting both dumps together (value = instance << 48 | epoch << 24 | session)
    K = np.concatenate([k0, k1])
    H = np.concatenate([v0 >> 48, v1 >> 48])
    tag = np.concatenate([np.zeros(n0, np.int8), np.ones(n1, np.int8)])
    o = np.lexsort((tag, H, K))
    same = (K[o][1:] == K[o][:-1]) & (H[o][1:] == H[o][:-1])
    stay = np.zeros(n0, bool)
    stay[o[:-1][same]] = True
    assert stay.sum() == n1 and np.array_equal(v0[stay], v1), "survivors are entries of the index, unchanged"
    # every entry that left precedes every entry that stayed under (epoch, key, instance)
    e0 = (v0 >> 24) & 0x3FFFFF
    def first(mask, last):
        idx = np.lexsort((H[:n0][mask], k0[mask], e0[mask]))
        j = idx[-1] if last else idx[0]
        return int(e0[mask][j]), int(k0[mask][j]), int(H[:n0][mask][j])
    assert first(~stay, True) < first(stay, False)
    say(f"  eviction: {n0} -> {n1} entries")
