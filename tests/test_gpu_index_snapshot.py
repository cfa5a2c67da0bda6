"""Whole-index snapshots through smetric_index_attach, and tables sized by an explicit
slot count (GPU, through the C ABI, against the oracle)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_08565_amd import workload as W
from tests.parity import Pair, run_sessions, say

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def test_snapshot_attach_restore():
    """A device copy of the index buffer, attached as a second index, holds exactly the
    entries of the original; the original moves on (routing, insert, eviction) while the
    copy stays put; restoring the original from the copy brings back the old entries,
    and the restored index routes the next batch as the oracle does from that state."""
    from paper_2607_08565_amd import smetric as S
    wl = W.config0(n_sess=32, n_turns=4)
    pair, _ = run_sessions(wl, 2, capacity=200_000)
    ok, ov = pair.oix.dump()
    n0 = pair.oix.size
    snap = pair.gix.snapshot()
    copy = S.Index.attach(snap, pair.gix.capacity, wl.n_inst)
    gk, gv = copy.dump()
    assert np.array_equal(gk, ok) and np.array_equal(gv, ov)
    assert copy.stats() == (n0, 0)
    # a too-short buffer or a different instance count cannot be attached
    with pytest.raises(S.SmetricError):
        S.Index.attach(snap[: snap.numel() // 2], pair.gix.capacity, wl.n_inst)
    with pytest.raises(S.SmetricError):
        S.Index.attach(snap, pair.gix.capacity, 0)
    # the original moves on; the copy does not
    b2 = wl.batch(2)
    pair.step(b2, what="batch 2 after the snapshot")
    pair.gix.evict(1, 4)
    assert pair.oix.evict(1, 4) == 0
    pair.compare_index("evicted after the snapshot")
    gk, gv = copy.dump()
    assert np.array_equal(gk, ok) and np.array_equal(gv, ov)
    # restore: the original equals the snapshot again, and routes batch 2 as an oracle
    # rebuilt from the same entries does
    pair.gix.restore(snap)
    gk, gv = pair.gix.dump()
    assert np.array_equal(gk, ok) and np.array_equal(gv, ov)
    fresh = oracle.Index(200_000, wl.n_inst)
    for t in range(2):  # the oracle's own history up to the snapshot
        bt = wl.batch(t)
        if t > 0:
            pb = wl.batch(t - 1)
            blk, keys = oracle.hash_blocks(pb.tokens, pb.tok_off, W.BLOCK, W.DEFAULT_SEED)
            fresh.insert(keys, blk, wl.placement[t - 1], pb.session, t - 1)
        blk, keys = oracle.hash_blocks(bt.tokens, bt.tok_off, W.BLOCK, W.DEFAULT_SEED)
        m = fresh.match(keys, blk)
        tg, _ = oracle.route(m, bt.prompt_len, bt.hist_len, bt.turn, bt.q, W.DEFAULT_PARAMS, bt.rr_base)
        fresh.insert(keys, blk, tg, bt.session, bt.epoch)
    fk, fv = fresh.dump()
    assert np.array_equal(fk, ok) and np.array_equal(fv, ov)
    pair.oix = fresh
    pair.step(wl.batch(2), what="batch 2 from the restored index")


@pytest.mark.parametrize("probed", [False, True])
def test_full_table_explicit_slots_with_eviction(probed):
    """A table sized by slot count to be ~15/16 full at capacity (the fullest allowed):
    closed-loop batches with shared prefixes (bitmap records), eviction after each batch
    -- in place while tombstones fit in half the free slots, then by rebuild -- every
    step's keys, rows, decisions and dump against the oracle."""
    wl = W.config3(n_sess=96, n_turns=5, prefix_len=2048, tail=(256, 2000), app=512)
    cap = 24_000  # the live entries reach ~23,300: the table ends ~0.88 full
    T = max(8, -(-wl.n_inst // 128))  # the spill threshold: keys with more holders get a bitmap record
    reserved = cap + T * min(max(64, cap // 256), cap // (T + 1) + 1)
    n_slots = -(-reserved * 16 // 15) + 8
    pair, br = run_sessions(wl, 5, capacity=cap, evict=(1, 20), probed=probed, n_slots=n_slots)
    assert pair.gix.n_slots < 8 * ((cap + 8 * max(64, cap // 256)) * 4 // 3 // 8)
    n, st = pair.gix.stats()
    say(f"explicit slots {pair.gix.n_slots}, entries {n}, occupancy {n / pair.gix.n_slots:.3f}")
    assert st == 0
