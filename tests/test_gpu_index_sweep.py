"""The whole path -- hash, match, route, post-route insert, LRU eviction -- against the
oracle on seeded random session workloads that vary everything at once: 1 to 300
instances, block sizes 2..64, prompts from empty to thousands of tokens over vocabularies
from 3 tokens to 2^31, up to three shared system prefixes, sessions that copy an earlier
one (pairs repeated within a batch), open-loop placements or closed-loop routing, every
load model, capacities from exact to loose, no eviction or 1/20 to all of the index
after every batch, the self-contained and the region-ordered (probed) insert.  Keys,
matched rows, targets, branches and the sorted index dump are compared bit for bit after
every step (tests/parity.py)."""
import numpy as np
import pytest

from paper_2607_08565_amd import workload as W
from tests.parity import Pair, say

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(dev):
    yield


def _workload(rng, case):
    n_inst = int(rng.choice([1, 2, 3, 7, 64, 65, 130, 300]))
    n_sess = int(rng.integers(1, 160))
    n_turns = int(rng.integers(2, 5))
    B = int(rng.choice([2, 16, 16, 64]))
    vocab = int(rng.choice([3, 1 << 20, 1 << 31]))
    lens = np.zeros((n_turns, n_sess), np.int64)
    lens[0] = rng.integers(0, 2000, n_sess)
    for t in range(1, n_turns):
        lens[t] = lens[t - 1] + rng.integers(0, 1500, n_sess)
    prefixes = [rng.integers(0, vocab, int(rng.choice([B * 3, 512, 1000]))).astype(np.int32)
                for _ in range(int(rng.integers(0, 4)))]
    streams = []
    for s in range(n_sess):
        tot = int(lens[-1, s])
        if s > 0 and rng.random() < 0.1:  # a copy of an earlier session
            head = streams[int(rng.integers(0, s))]
        elif prefixes and rng.random() < 0.6:
            head = prefixes[int(rng.integers(0, len(prefixes)))]
        else:
            head = np.zeros(0, np.int32)
        st = np.concatenate([head, rng.integers(0, vocab, max(0, tot - len(head)))]).astype(np.int32)
        streams.append(st)
    lens = np.minimum(lens, np.array([len(s) for s in streams])[None, :])
    placement = rng.integers(0, n_inst, (n_turns, n_sess)).astype(np.int32) if rng.random() < 0.5 else None
    wl = W.SessionWorkload(5000 + case, n_inst, n_sess, n_turns, lens, streams,
                           str(rng.choice(["uniform100", "poisson50", "prev_counts"])), placement)
    return wl, B


@pytest.mark.parametrize("chunk", range(4))
def test_path_on_random_session_workloads(chunk):
    for case in range(74000 + 10 * chunk, 74000 + 10 * (chunk + 1)):
        rng = np.random.default_rng(case)
        wl, B = _workload(rng, case)
        open_loop = wl.placement is not None
        blocks = int((wl.lens // B).sum()) * (2 if open_loop else 1)
        capacity = max(16, int(blocks * float(rng.choice([1.0, 1.5, 3.0]))) + 8)
        evict = [None, (1, 20), (1, 8), (1, 3), (1, 1), (0, 1)][int(rng.integers(0, 6))]
        probed = bool(rng.random() < 0.5)
        say(f"  case {case}: I={wl.n_inst} S={wl.n_sess} T={wl.n_turns} B={B} open={open_loop} "
            f"capacity={capacity} evict={evict} probed={probed}")
        pair = Pair(capacity, wl.n_inst, block=B)
        params = dict(W.DEFAULT_PARAMS, block_size=B)
        prev = None
        for t in range(wl.n_turns):
            if open_loop and t > 0:
                pb = wl.batch(t - 1)
                d_boff, nb, d_keys, okeys, blk_off = pair.hash_both(pb.tokens, pb.tok_off)
                assert pair.insert_both(d_keys, d_boff, nb, okeys, blk_off, wl.placement[t - 1], pb.session,
                                        t - 1) == 0
            prev, _ = pair.step(wl.batch(t, prev), params=params, what=f"case {case} batch {t}", probed=probed)
            if evict is not None:
                pair.gix.evict(*evict)
                assert pair.oix.evict(*evict) == 0
                pair.compare_index(f"case {case} batch {t} after evict")
