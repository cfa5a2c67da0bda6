"""GPU LRU eviction (through the C ABI) vs the CPU oracle, bit for bit on the dumped entry
set: fractions 0, small, large and 1 of the entries; many entries sharing one epoch (the
key decides), keys held by many instances (the instance decides) including keys held by
more than the holder-list threshold (bitmap records, rebuilt after the eviction), and
inserts between evictions into the rebuilt table."""
import numpy as np
import pytest
import torch

import oracle
from tests.parity import Pair, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def _insert(pair, rng, pool, n_req, per_req, n_inst, epoch):
    """n_req requests, each a random subset of `pool` (distinct keys), each on a random
    instance; the same keys recur across requests and epochs."""
    ks = [rng.choice(pool, size=int(rng.integers(1, per_req + 1)), replace=False) for _ in range(n_req)]
    okeys = np.concatenate(ks).astype(np.uint64)
    blk_off = np.zeros(n_req + 1, np.int64)
    blk_off[1:] = np.cumsum([len(k) for k in ks])
    inst = rng.integers(0, n_inst, n_req).astype(np.int32)
    sess = rng.integers(0, 1 << 24, n_req).astype(np.uint32)
    d_keys = torch.from_numpy(okeys.view(np.int64)).cuda().view(torch.uint64)
    rc = pair.insert_both(d_keys, to_dev(blk_off), int(blk_off[-1]), okeys, blk_off, inst, sess, epoch)
    assert rc == 0


def test_evict_fractions_ties_and_hot_keys():
    rng = np.random.default_rng(11)
    n_inst = 40  # holder-list threshold 8: keys on more instances get bitmap records
    pair = Pair(300_000, n_inst)
    pool = rng.integers(1, 2**63, 4000, dtype=np.int64).astype(np.uint64)
    hot = pool[:16]  # in every request: held by (nearly) every instance
    for epoch in range(4):
        _insert(pair, rng, pool, 300, 60, n_inst, epoch)
        hk = np.tile(hot, 40).astype(np.uint64)
        blk_off = np.arange(0, len(hk) + 1, len(hot), dtype=np.int64)
        d_keys = torch.from_numpy(hk.view(np.int64)).cuda().view(torch.uint64)
        assert pair.insert_both(d_keys, to_dev(blk_off), len(hk), hk, blk_off, np.arange(40, dtype=np.int32),
                                np.full(40, 7, np.uint32), epoch) == 0
    pair.compare_index("before eviction")
    for t, (num, den) in enumerate([(0, 5), (1, 20), (1, 3), (7, 9), (1, 1)]):
        n0, _ = pair.gix.stats()
        pair.gix.evict(num, den)
        assert pair.oix.evict(num, den) == 0
        pair.compare_index(f"evict {num}/{den}")
        n1, _ = pair.gix.stats()
        assert n0 - n1 == -(-n0 * num // den)
        say(f"  evict {num}/{den}: {n0} -> {n1}")
        _insert(pair, rng, pool, 200, 40, n_inst, 10 + t)  # the rebuilt table takes inserts
        pair.compare_index(f"insert after evict {num}/{den}")


def test_evict_one_epoch_instance_ties():
    """Every entry in one epoch and every key on many instances: the cut falls between
    instances of one key, decided by the last digits of the selection."""
    rng = np.random.default_rng(12)
    pair = Pair(100_000, 300)
    pool = rng.integers(1, 2**63, 50, dtype=np.int64).astype(np.uint64)
    for _ in range(3):
        _insert(pair, rng, pool, 400, 50, 300, 5)
    n0, _ = pair.gix.stats()
    for num, den in [(1, 7), (1, 2), (2, 3)]:
        pair.gix.evict(num, den)
        assert pair.oix.evict(num, den) == 0
        pair.compare_index(f"evict {num}/{den}")
    say(f"  {n0} entries, one epoch")
